"""Static checks of the C ABI's ownership rules (no GPU needed).

The header promises that only create calls (and the set-up call
tgm_state_set_mitigation) allocate device memory or synchronise the device,
so that per-batch calls and the pipelined executor never stall the GPU.
These checks read the library's sources: every device allocation goes
through the counting wrapper, and the functions that allocate, create
events or synchronise the device are set-up functions, reached only from
set-up calls.  The GPU side of the same promise (the allocation count does
not move across tgm_stage_run) is in tests/test_gpu_executor_trace.py.
"""
import glob
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2402_15113_amd", "csrc")

# set-up functions that may allocate, create events or synchronise the device
SETUP = {"tgm_graph_create", "tgm_state_create", "tgm_model_create", "create_jodie",
         "tgm_trainer_create", "tgm_apan_create",
         "tgm_mitigator_create", "mitigate_reserve", "tgm_state_set_mitigation",
         "tgm_state_save", "tgm_state_restore", "tgm_state_load", "tgm_state_read",
         "upload", "tgm_profile_get", "tgm_profile_count", "fold_profile", "take_event",
         "tgm_noalloc_init", "static_scratch_ptr", "gru_w_setup"}
SETUP_CALLERS = {"mitigate_reserve": {"tgm_mitigator_create", "tgm_state_set_mitigation"},
                 "gru_w_setup": {"tgm_model_create", "create_jodie"}}
FORBIDDEN = re.compile(r"\b(dev_malloc|hipMalloc\w*|hipDeviceSynchronize|hipEventCreate\w*|"
                       r"hipMemset|hipStreamSynchronize|hipHostMalloc|hipFree)\s*\(")


def all_function_bodies():
    """Like functions(), but descends into namespace { } blocks."""
    res = []
    for path in sorted(glob.glob(os.path.join(CSRC, "*.hip"))):
        text = open(path).read()
        text = re.sub(r"//[^\n]*", "", text)
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        text = re.sub(r'"(\\.|[^"\\])*"', '""', text)
        res += _scan(os.path.basename(path), text)
    return res


def _scan(fname, text):
    out = []
    k, n, head_from = 0, len(text), 0
    while k < n:
        ch = text[k]
        if ch == ";" or ch == "}":
            head_from = k + 1
        elif ch == "{":
            head = text[head_from:k]
            depth, j = 1, k + 1
            while depth and j < n:
                depth += {"{": 1, "}": -1}.get(text[j], 0)
                j += 1
            body = text[k + 1:j - 1]
            last = head.strip()
            if re.search(r"\bnamespace\b[^()]*$", last) or re.search(r'extern\s*""\s*$', last):
                out += _scan(fname, body)
            else:
                m = re.search(r"([A-Za-z_][\w:]*)\s*\((?:[^()]|\([^()]*\))*\)\s*(const\s*)?$",
                              last, re.S)
                if m:
                    out.append((fname, m.group(1).split("::")[-1], body))
            k, head_from = j, j
            continue
        k += 1
    return out


def test_every_device_allocation_is_counted():
    for path in glob.glob(os.path.join(CSRC, "*")):
        text = re.sub(r"//[^\n]*", "", open(path).read())
        for m in re.finditer(r"\bhipMalloc\w*\s*\(", text):
            line = text[:m.start()].count("\n") + 1
            assert path.endswith("common.h"), f"{path}:{line} allocates outside dev_malloc"


def test_only_setup_functions_allocate_or_synchronise():
    fns = all_function_bodies()
    assert len(fns) > 50
    names = {n for _, n, _ in fns}
    for must in ("tgm_stage_run", "compute_iteration", "tgm_update_memory", "tgm_embed",
                 "tgm_fetch_memory", "tgm_sample_nodes", "tgm_state_create"):
        assert must in names, must
    for fname, name, body in fns:
        hits = sorted({m.group(1) for m in FORBIDDEN.finditer(body)})
        if hits and not name.endswith("_destroy") and name not in SETUP:
            raise AssertionError(f"{fname}: {name} calls {hits} but is not a set-up function")


def test_setup_helpers_are_reached_only_from_setup_calls():
    fns = all_function_bodies()
    for helper, allowed in SETUP_CALLERS.items():
        for fname, name, body in fns:
            if name != helper and re.search(rf"\b{helper}\s*\(", body):
                assert name in allowed, f"{fname}: {name} calls {helper}"


def test_executor_creates_nothing():
    body = [b for f, n, b in all_function_bodies() if n == "tgm_stage_run"]
    assert len(body) == 1
    assert not re.search(r"\b(hipEventCreate|hipStreamCreate|dev_malloc|hipMalloc|new\s)", body[0])


def test_citations():
    """The staleness mitigation is Sec. 3.3 (Sec. 4 is the theoretical
    analysis and has no subsections)."""
    pats = re.compile(r"Sec\.\s*4\.\d|App\.\s*C\.3\b.*(gap|Δt|staleness error)")
    for path in (glob.glob(os.path.join(ROOT, "paper_2402_15113_amd", "**", "*.*"), recursive=True)
                 + glob.glob(os.path.join(ROOT, "oracle", "*.*"))
                 + glob.glob(os.path.join(ROOT, "include", "*.h"))
                 + glob.glob(os.path.join(ROOT, "tests", "*.py"))
                 + [os.path.join(ROOT, "DESIGN.md"), os.path.join(ROOT, "bench.py")]):
        if path.endswith((".so", ".o", ".pyc")) or os.path.basename(path) == "test_boundary.py":
            continue
        try:
            text = open(path, encoding="utf-8").read()
        except (UnicodeDecodeError, IsADirectoryError):
            continue
        for k, line in enumerate(text.splitlines(), 1):
            assert not pats.search(line), f"{path}:{k}: {line.strip()}"
