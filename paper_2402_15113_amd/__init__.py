"""MI355X (gfx950) implementation of the per-batch memory-module stage of
memory-based temporal GNN training (MSPipe, KDD'24): HIP kernels behind the C
ABI of include/tgm.h (libtgm.so), a ctypes binding with the same names
(``tgm``) and a stage runner (``stage.Stage``).  Importing the package loads
nothing; ``tgm.lib()`` loads the library and fails if it is not built."""

__all__ = ["tgm", "stage"]
