// Internal interface between the C-ABI host layer (ssd_api.cpp) and the
// kernel launchers (ssd_*.hip).  Not installed; not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ssd {

// Internal choices a test or a measurement may override for the whole process
// (ssd_set_tuning in the C ABI; every value 0 = the library's own choice).
enum Tuning {
    kTuneForceGeneral = 0,   // 1: the general step-by-step kernels for every call
    kTuneHeadsPerItem,       // heads per work item of the fused chunk kernel
    kTuneEarlyFlag,          // 1: state flag after the output stage, 2: right after the state store
    kTuneMaxWorkgroups,      // cap on the fused chunk kernel's persistent workgroups
    kTuneSeparatePost,       // 1: gate and normalisation always in their own output pass
    kTuneBwdHeadsPerSlice,   // heads per workgroup of the backward's chunk kernel
    kTuneVarlenPerSequence,  // 1: packed rows by host offsets run one call per sequence
    kTuneStateWaitLimit,     // polls before a chunk's wait for the state before it gives up
    kTuneFusedRightFactor,   // 1: the chunk kernel's right factor in its own pass, 2: in the diagonal block's
    kTunePackedOrder,        // 1: a packed row's chunks taken in table order, 2: by index within their sequence
    kTuneCount
};
int64_t tuning(Tuning k);

// Polls (each followed by a short sleep) before a chunk kernel's wait for the
// state of the chunk before it gives up and reports SSD_ERR_STATE_TIMEOUT.
constexpr int64_t kDefaultSpinLimit = 1LL << 22;

// Every workspace begins with a 256-byte header; its first int is the status
// word of the last forward that used it (0 = fine, 1 = a state wait gave up).
constexpr size_t kWorkspaceHeader = 256;

// dt parameterisation of the block path: dt = clamp(softplus?(dt_in + bias)).
// `active` false = dt is used as given (the plain layer).
struct DtTransform {
    const float* bias = nullptr;   // (H) or null
    int softplus = 0;
    float lo = 0.f, hi = 0.f;
    bool active = false;
};

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
    DtTransform dtx;
    int* status = nullptr;   // status word, zeroed by the first kernel when not null
};

struct WorkspaceLayout {
    size_t cs, info, gram, states, total;
};

WorkspaceLayout workspace_layout(int64_t b, int64_t H, int64_t P, int64_t N, int64_t G,
                                 int64_t Q, int64_t nC);

// Enqueue the whole forward on `stream`; returns the first launch or record
// error.  `ev_begin` / `ev_end` (may be null) are recorded on `stream` right
// before and right after the dominant kernel (the chunk-output kernel here,
// the chunk kernel of the fused path).
hipError_t launch_unfused(const Params& p, bool bf16, hipStream_t stream,
                          hipEvent_t ev_begin, hipEvent_t ev_end);

// Fused path (bf16, P = 64, N in {64, 128, 256}, Q = 256; plain rows or one packed row).
// Sequence starts of a packed row handed to the device by value (kernel
// argument) when the caller gives them in host memory: n sequences, v[0..n].
constexpr int kArgSeqs = 511;
struct SeqStartsArg {
    int n;
    int v[kArgSeqs + 1];
};

struct FusedParams {
    int64_t b, T, H, P, N, G, nC, HG;
    const void* x;
    const void* dt;
    const float* A_log;
    const void* B;
    const void* C;
    const float* D;
    const float* init;
    void* y;
    float* fin;
    // workspace
    uint16_t* gram;   // (b, G, nC, tiles, 64 lanes, 4) causal Gram tiles, bf16, per-lane layout
    uint16_t* BT;     // (b, G, nC, N, Q) B^T per chunk, bf16
    float* ring;      // (b, H, 2, P, N) chunk-state ring
    int* flags;       // (b, H, nC)      state-published flags
    int* ticket;      // [0] work ticket, [2] chunk table entries of a packed row
    int* status;      // set to 1 when a state wait gives up (zeroed first when reset_status)
    int reset_status = 1;
    int64_t spin_limit = kDefaultSpinLimit;
    int max_workgroups = 0;   // > 0: cap on the chunk kernel's persistent workgroups
    DtTransform dtx;
    // Packed row (batch 1) with device seq_idx: every sequence is cut into
    // chunks of its own (the last one partial), listed in token order in a
    // device table that k_seq_chunks builds; nC is then the table's capacity.
    // Null seq_idx: plain rows, chunk c of row b at token c Q.
    const int32_t* seq_idx = nullptr;  // (T)
    const SeqStartsArg* arg_starts = nullptr;  // host memory, instead of seq_idx; read at launch
    int64_t nseq = 0;
    int* starts = nullptr;             // (nseq + 1) first token of each sequence, then T
    int4* vtab = nullptr;              // (nC) {first token, length, sequence, bit 0 first chunk of
                                       //  its sequence | bit 1 last | ring row << 2}
    int* vcount = nullptr;             // [0] table entries
    // (nC) the order in which the chunk kernel takes the table's entries
    // (null: table order); see k_seq_order
    int* vorder = nullptr;
    int64_t ring_rows = 0;             // sequences of more than one chunk that the ring holds
    // nonzero: a chunk's state flag is set as soon as its state is stored
    // (before its left factor), for launches bound by the chain of chunks
    int early_flag = 0;
    // nonzero: the right factor (the first column block's, with two) is
    // computed in the diagonal block's pass over x (plain rows, late flag)
    int fuse_rf = 0;
    // gate / per-head normalisation in the output stage (null: none)
    const void* z = nullptr;             // (b, T, H, P) bf16
    const float* norm_weight = nullptr;  // (H * P), with norm_head
    int norm_head = 0;                   // nonzero: RMS-normalise each head's P channels
    float norm_eps = 0.f;
    // nonzero: y is float32 (plain rows, no gate or normalisation)
    int y32 = 0;
};

struct FusedLayout {
    size_t gram, BT, ring, flags, ticket, starts, vtab, vorder, total;
    int64_t nC;          // chunks the layout holds (table capacity for a packed row)
    int64_t ring_rows;   // rows of the state ring
};

int64_t heads_per_workgroup(int64_t heads_per_group, int64_t items_per_head, int compute_units);
bool fused_supported(int64_t P, int64_t N, int64_t Q, bool bf16);
// The chunk table of a packed row of T tokens and nseq sequences, from the
// device seq_idx or, when it is null, from starts handed over by value: every
// sequence cut into chunks of Q tokens (256 or 64) from its first token on,
// at most `cap` entries; seq_first (may be null) gets each sequence's first
// entry and then the entry count.  `starts` is (nseq + 1) ints of workspace.
hipError_t launch_seq_table(const int32_t* seq_idx, const SeqStartsArg* arg_starts, int64_t T, int64_t nseq, int Q,
                            int64_t cap, int64_t ring_rows, int* starts, int4* vtab, int* seq_first, int* vcount,
                            hipStream_t stream);
// nseq > 0: layout for one packed row of nseq sequences (seq_idx); nC is the
// row's chunk count ceil(T / Q) either way.
FusedLayout fused_layout(int64_t b, int64_t T, int64_t H, int64_t N, int64_t G, int64_t nC, int64_t nseq);
hipError_t launch_fused(const FusedParams& p, hipStream_t stream, hipEvent_t ev_begin,
                        hipEvent_t ev_end);

// Decode step (one token per sequence, state updated in place).
struct DecodeParams {
    int64_t b, H, P, N, G;
    const void* x;      // (b, H, P)
    const void* dt;     // (b, H)
    const float* A_log;
    const void* B;      // (b, G, N)
    const void* C;      // (b, G, N)
    const float* D;     // (H) or null
    float* state;       // (b, H, P, N)
    void* y;            // (b, H, P)
};

hipError_t launch_decode(const DecodeParams& p, bool bf16, hipStream_t stream);

// Gate and grouped RMS normalisation of the block, in place on y (b*T token
// rows of H*P channels): y = y * silu(z) when z, then the normalisation over
// groups of `group` channels (a multiple of P) when group > 0.
struct GateNormParams {
    int64_t rows, C, group;
    void* y;
    const void* z;             // or null
    const float* weight;       // (C) or null
    float eps;
};

hipError_t launch_gate_norm(const GateNormParams& p, bool bf16, hipStream_t stream);

// Sequence spans (context parallelism).
struct SpanParams {
    int64_t b, T, H, P, N, G, nC;   // T: the span's length; nC: its 256-token chunks
    const void* dt;                 // (b, T, H)
    const float* A_log;
    const void* C;                  // (b, T, G, N)
    const float* entering;          // (b, H, P, N)
    void* y;                        // (b, T, H, P), updated in place
    float* sums;                    // workspace (b, H, nC): dt sums per chunk
};

int64_t span_chunks(int64_t T);
hipError_t launch_span_decay(int64_t b, int64_t T, int64_t H, const void* dt, const float* A_log, float* decay,
                             bool bf16, hipStream_t stream);
hipError_t launch_span_combine(int64_t R, int64_t bh, int64_t PN, const float* decay, const float* local,
                               const float* init, float* entering, float* fin, hipStream_t stream);
hipError_t launch_span_correct(const SpanParams& p, bool bf16, hipStream_t stream);

}  // namespace ssd
