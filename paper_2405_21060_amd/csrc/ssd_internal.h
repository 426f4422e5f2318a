// Internal interface between the C-ABI host layer (ssd_api.cpp) and the
// kernel launchers (ssd_*.hip).  Not installed; not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ssd {

// One call's shapes, pointers and workspace carve-up.
struct Params {
    int64_t b, T, H, P, N, G, Q, nC, nseq;
    const void* x;
    const void* dt;
    const float* A_log;
    const void* B;
    const void* C;
    const float* D;
    const float* init;
    const int32_t* seq_idx;
    void* y;
    float* fin;
    // workspace
    float* cs;       // (b, H, nC, Q)  chunk-local inclusive cumsum of dt*A, log2 units
    int4* info;      // (b, H, nC)     per-chunk scan coefficients (see ssd_unfused.hip)
    float* gram;     // (b, G, nC, Q, Q) C B^T per chunk (lower block triangle only)
    float* states;   // (b, nC, H, P, N) chunk states, then states entering each chunk
};

struct WorkspaceLayout {
    size_t cs, info, gram, states, total;
};

WorkspaceLayout workspace_layout(int64_t b, int64_t H, int64_t P, int64_t N, int64_t G,
                                 int64_t Q, int64_t nC);

// Enqueue the whole forward on `stream`; returns the first launch error.
hipError_t launch_unfused(const Params& p, bool bf16, hipStream_t stream);

}  // namespace ssd
