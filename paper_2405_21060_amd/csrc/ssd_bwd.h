// Internal interface of the backward kernels (ssd_backward.hip) for the C-ABI
// host layer.  Not installed; not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ssd {

// Tokens per chunk of the backward's own decomposition (independent of the
// forward's chunk size: the gradient of the layer does not depend on it):
// 32 on the general path, 64 on the matrix-core path.
constexpr int64_t kBwdQ = 32;
constexpr int64_t kBwdQFast = 64;

struct BwdParams {
    int64_t b, T, H, P, N, G, nC;   // nC = ceil(T / chunk) (kBwdQ, or kBwdQFast)
    int64_t S, hs;                  // head slices per group, heads per slice
    const void* x;
    const void* dt;
    const float* A_log;
    const void* B;
    const void* C;
    const float* D;        // may be null
    const float* init;     // may be null
    const void* dy;
    const float* dfinal;   // may be null
    void* dx;
    void* ddt;
    float* dA_log;
    void* dB;
    void* dC;
    float* dD;             // may be null
    float* dinit;          // may be null
    // workspace (float32)
    float* cs;     // (b, H, nC, kBwdQ)   chunk-local inclusive cumsum of dt*A, log2 units
                   //                     (general path only)
    float* hin;    // (b, nC, H, P, N)    chunk states, then the state entering each chunk
                   //                     (matrix-core path: bf16, (b, nC, H, N, P))
    float* gn;     // (b, nC, H, P, N)    output-to-state terms, then the gradient of the state
                   //                     leaving each chunk (general path only)
    float* gnT;    // matrix-core path only: the same, transposed, bf16 (b, nC, H, N, P)
    float* dBp;    // (S, b, T, G, N)     dB over one slice of a group's heads
    float* dCp;    // (S, b, T, G, N)
    float* dAp;    // (b, H, nC)          per-chunk terms of dA
    float* dDp;    // (b, H, nC)          per-chunk terms of dD
    // Packed row (b = 1, matrix-core path): every sequence cut into chunks of
    // its own; nC is then the chunk table's capacity.  Null vtab: plain rows.
    int64_t nseq = 0;
    const int4* vtab = nullptr;     // (nC) {first token, length, sequence, flags}
    const int* seq_first = nullptr; // (nseq + 1) first table entry of each sequence, then the count
    const int* vcount = nullptr;    // [0] table entries
    // Matrix-core path, plain rows: nonzero = dt and dy are float32 and ddt is
    // written in float32 (the block gradients' handoffs); x, B, C, dx, dB, dC
    // keep the bf16 activation dtype.
    int h32 = 0;
    // matrix-core path, one head slice per group (S == 1) and dB, dC 8-byte
    // aligned: the chunk kernel stores dB and dC (bf16) itself; set at launch
    int bc_direct = 0;
};

struct BwdLayout {
    size_t cs, hin, gn, gnT, dBp, dCp, dAp, dDp, total;
};

// Head slices: enough (b, chunk, group, slice) workgroups to fill the chip.
void bwd_slices(int64_t b, int64_t nC, int64_t G, int64_t heads_per_group, int64_t* S, int64_t* hs);

BwdLayout bwd_layout(int64_t b, int64_t T, int64_t H, int64_t P, int64_t N, int64_t G, int64_t nC, int64_t S,
                     bool fast);

// The matrix-core path covers bf16 with headdim 64 and dstate 64 or 128.
bool bwd_fast_supported(bool bf16, int64_t P, int64_t N);
hipError_t launch_backward_fast(const BwdParams& p, hipStream_t stream, hipEvent_t ev_begin, hipEvent_t ev_end);

// The final sums over head slices (dB, dC) and over rows and chunks (dA_log,
// dD), shared by both paths; with with_bc false only the latter (the chunk
// kernel stored dB and dC itself).
hipError_t launch_backward_reduce(const BwdParams& p, bool bf16, hipStream_t stream, bool with_bc = true);

// out[c] = sum over r of part[r * ncols + c], r in order (float32).
hipError_t launch_sum_rows(const float* part, int64_t nrows, int64_t ncols, float* out, hipStream_t stream);

// Enqueue the whole backward on `stream`; `ev_begin` / `ev_end` (may be null)
// are recorded right before and right after the chunk-gradient kernel.
hipError_t launch_backward(const BwdParams& p, bool bf16, hipStream_t stream, hipEvent_t ev_begin,
                           hipEvent_t ev_end);

}  // namespace ssd
