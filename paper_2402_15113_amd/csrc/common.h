// Internal declarations shared by the libtgm translation units (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <vector>

#include "tgm.h"

namespace tgm {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// ---------------------------------------------------------------- errors
void record_error(hipError_t e);

#define TGM_HIP(call)                                  \
    do {                                               \
        hipError_t e_ = (call);                        \
        if (e_ != hipSuccess) {                        \
            ::tgm::record_error(e_);                   \
            return TGM_EDEVICE;                        \
        }                                              \
    } while (0)

#define TGM_LAUNCHED()                                 \
    do {                                               \
        hipError_t e_ = hipGetLastError();             \
        if (e_ != hipSuccess) {                        \
            ::tgm::record_error(e_);                   \
            return TGM_EDEVICE;                        \
        }                                              \
    } while (0)

inline hipStream_t as_stream(void *s) { return reinterpret_cast<hipStream_t>(s); }

// Per-kernel timing (tgm_profile_*): prof_begin returns -1 when disabled.
int prof_begin(const char *kernel, hipStream_t s);
void prof_end(int id, hipStream_t s);

// Launch a kernel, timed when profiling is on, and check the launch.
#define TGM_LAUNCH(kern, grid, block, lds, s, ...)                       \
    do {                                                                 \
        const int pid_ = ::tgm::prof_begin(#kern, s);                    \
        hipLaunchKernelGGL(kern, grid, block, lds, s, __VA_ARGS__);      \
        ::tgm::prof_end(pid_, s);                                        \
        TGM_LAUNCHED();                                                  \
    } while (0)

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int32_t round_up(int32_t a, int32_t b) { return (int32_t)cdiv(a, b) * b; }

// ---------------------------------------------------------------- handles
// One adjacency entry: an event touching the node, with its time and the
// other endpoint.  16 bytes, so the k entries a sampler reads are one
// contiguous 16k-byte run.
struct AdjRec {
    double ts;
    int32_t eid;
    int32_t nbr;
};

}  // namespace tgm

struct tgm_graph {
    int32_t N = 0;
    int64_t E = 0;
    int32_t D_e = 0;
    const int32_t *src = nullptr, *dst = nullptr, *neg = nullptr;
    const double *t = nullptr;
    const float *efeat = nullptr;
    int64_t *off = nullptr;           // [N + 1]
    tgm::AdjRec *adj = nullptr;       // [n_adj]
    int64_t n_adj = 0;
};

struct tgm_state {
    int32_t N = 0, M = 0, D_m = 0, s = 0, max_batch = 0;
    // committed tables
    float *mem = nullptr, *mail = nullptr;
    double *mem_ts = nullptr, *mail_ts = nullptr;
    int32_t *ver = nullptr;
    // ring of s + 1 staged write sets, each indexed by candidate c in [0, 2b):
    // candidate c is (event first + c/2, role c%2)
    int32_t *r_flag = nullptr, *r_node = nullptr;
    float *r_mem = nullptr, *r_mail = nullptr;
    double *r_mem_ts = nullptr, *r_mail_ts = nullptr;
    struct Slot {
        int64_t iter = -1;
        int32_t b = 0;
        bool staged = false;
    };
    std::vector<Slot> ring;
    int64_t committed_through = -1;   // all writes <= this are in the tables
    int64_t staged_through = -1;      // last iteration whose update was issued
    int64_t last_fetch = INT64_MIN;
    int32_t *win = nullptr;           // [N] latest candidate per node-set position
    size_t ring_rows() const { return 2 * (size_t)max_batch; }
};

struct tgm_model {
    int32_t M = 0, D_e = 0, D_t = 0, H = 0, nb = 0, max_nodes = 0, max_roots = 0;
    int32_t D_m = 0, D_x = 0;
    // GRU: packed B operands and biases
    int32_t KXC = 0, KHC = 0, MB = 0;   // 16-wide chunks of D_x, M and hidden blocks
    tgm::f4 *gru_bx = nullptr;           // [3][KXC][MB][64]
    tgm::f4 *gru_bh = nullptr;           // [3][KHC][MB][64]
    float *gru_bias = nullptr;           // [4][MB*16]: b_ir+b_hr, b_iz+b_hz, b_in, b_hn
    double *omega = nullptr, *beta = nullptr;
    // node projections P = s' [W_q^s; W_k^s; W_v^s]^T
    int32_t PC = 0, PNB = 0;             // chunks of M, 16-col blocks of 3M
    tgm::f4 *proj_b = nullptr;
    float *P = nullptr;                  // [max_nodes x PNB*16]
    // attention: per-slot part [efeat || phi] -> [K | V]
    int32_t KFC = 0, KVNB = 0;           // chunks of D_e + D_t, 16-col blocks of 2M
    tgm::f4 *kv_b = nullptr;
    float *b_k = nullptr, *b_v = nullptr, *c_q = nullptr;   // [M] each
    // output projection
    int32_t OC = 0, ONB = 0;             // chunks of 2M, 16-col blocks of M
    tgm::f4 *out_b = nullptr;
    float *b_o = nullptr;
};

namespace tgm {

// ---------------------------------------------------------------- device
// v_mfma_f32_16x16x4_f32: lane l supplies A[l%16][l/16] and B[l/16][l%16];
// the 4 results of lane l are C[4*(l/16) + v][l%16], v = 0..3.
__device__ __forceinline__ f4 mfma_16x16x4(float a, float b, f4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// 16 consecutive k of one 16x16 output block.  Lane l holds a = A[row][k0 + 4q
// .. +3] and b = B[k0 + 4q .. +3][col] with q = l/16, row = col = l%16; the
// four instructions each cover the k-slice {k0 + 4q + j}.
__device__ __forceinline__ f4 mfma_k16(f4 a, f4 b, f4 c)
{
    c = mfma_16x16x4(a.x, b.x, c);
    c = mfma_16x16x4(a.y, b.y, c);
    c = mfma_16x16x4(a.z, b.z, c);
    c = mfma_16x16x4(a.w, b.w, c);
    return c;
}

// Cosine time encoding with the phase formed in fp64: time gaps reach 1e8 s,
// where an fp32 phase would be off by whole radians.
__device__ __forceinline__ float time_enc(double omega, double beta, double dt)
{
    return (float)cos(fma(omega, dt, beta));
}

__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
        v += __shfl_xor(v, o, kWave);
    return v;
}

// Copy `n` floats with one wavefront; 16-byte accesses when both rows allow it.
__device__ __forceinline__ void wave_copy_row(float *__restrict__ dst,
                                              const float *__restrict__ src, int n, int lane)
{
    if (((reinterpret_cast<uintptr_t>(dst) | reinterpret_cast<uintptr_t>(src)) & 15) == 0 &&
        (n & 3) == 0) {
        const f4 *s4 = reinterpret_cast<const f4 *>(src);
        f4 *d4 = reinterpret_cast<f4 *>(dst);
        for (int k = lane; k < (n >> 2); k += kWave)
            d4[k] = s4[k];
    } else if (((reinterpret_cast<uintptr_t>(dst) | reinterpret_cast<uintptr_t>(src)) & 7) ==
                   0 &&
               (n & 1) == 0) {
        const f2 *s2 = reinterpret_cast<const f2 *>(src);
        f2 *d2 = reinterpret_cast<f2 *>(dst);
        for (int k = lane; k < (n >> 1); k += kWave)
            d2[k] = s2[k];
    } else {
        for (int k = lane; k < n; k += kWave)
            dst[k] = src[k];
    }
}

// ---------------------------------------------------------------- host
// Pack the B operand of C = A * W^T (W is n_out x K, row stride ldw, columns
// [c0, c0 + K)) for mfma_k16: out[((kc * NB + nb) * 64 + lane) * 4 + j] =
// W[16 nb + lane%16][c0 + 16 kc + 4 (lane/16) + j], zero outside.
std::vector<float> pack_b(const float *W, int n_out, int ldw, int c0, int K, int KC, int NB);

tgm_status_t upload(void *dst, const void *src, size_t bytes);

}  // namespace tgm
