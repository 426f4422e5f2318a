// C ABI of the SSD forward: validation, workspace planning, launch.
// Everything here runs on the host; no HIP call is made before the arguments
// have been validated, so an error return never leaves work on the stream.
#include "ssd.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <mutex>

#include "ssd_block_bwd.h"
#include "ssd_bwd.h"
#include "ssd_internal.h"

namespace ssd {

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

struct Shape {
    int64_t b, T, H, P, N, G, Q, nC, nseq;
    bool bf16;
};

// 2^31 - 1: every per-tensor element count must stay below it, and every
// kernel grid dimension far below it.
constexpr int64_t kMaxElems = 0x7fffffffLL;

int validate(const ssd_problem* prob, bool has_seq_idx, Shape* s)
{
    if (!prob) return SSD_ERR_NULL_ARG;
    if (prob->dtype != SSD_DTYPE_F32 && prob->dtype != SSD_DTYPE_BF16) return SSD_ERR_BAD_DTYPE;
    if (prob->batch < 1 || prob->seqlen < 1 || prob->nheads < 1 || prob->headdim < 1 ||
        prob->dstate < 1 || prob->ngroups < 1 || prob->nheads % prob->ngroups != 0)
        return SSD_ERR_BAD_SHAPE;
    const int64_t Q = prob->chunk_size;
    if (Q != 32 && Q != 64 && Q != 128 && Q != 256) return SSD_ERR_BAD_CHUNK;
    if (prob->headdim % 16 != 0 || prob->headdim > 128 || prob->dstate % 16 != 0 ||
        prob->dstate > 256)
        return SSD_ERR_UNSUPPORTED_DIMS;
    if (has_seq_idx) {
        if (prob->batch != 1) return SSD_ERR_SEQIDX_BATCH;
        if (prob->nseq < 1 || prob->nseq > prob->seqlen) return SSD_ERR_BAD_SHAPE;
    }
    s->b = prob->batch;
    s->T = prob->seqlen;
    s->H = prob->nheads;
    s->P = prob->headdim;
    s->N = prob->dstate;
    s->G = prob->ngroups;
    s->Q = Q;
    s->nC = (s->T + Q - 1) / Q;
    s->nseq = has_seq_idx ? prob->nseq : s->b;
    s->bf16 = prob->dtype == SSD_DTYPE_BF16;
    // index-range limits (grid y/z are H and b; flat element counts in int64
    // arithmetic everywhere, but keep each tensor addressable by 31 bits of
    // 16-byte vectors and the grid inside HIP's limits)
    if (s->H > 65535 || s->b > 65535 || s->nC > 0x7fffffff) return SSD_ERR_TOO_LARGE;
    const double elems_x = static_cast<double>(s->b) * s->T * s->H * s->P;
    const double elems_st = static_cast<double>(s->b) * s->nC * s->H * s->P * s->N;
    if (elems_x > 16.0 * kMaxElems || elems_st > 16.0 * kMaxElems) return SSD_ERR_TOO_LARGE;
    return SSD_OK;
}

}  // namespace

constexpr int64_t kMaxElemsPublic = kMaxElems;

// Process-wide overrides of internal choices (ssd_set_tuning); 0 = automatic.
namespace {
std::atomic<int64_t> g_tuning[kTuneCount];
}

int64_t tuning(Tuning k) { return g_tuning[k].load(std::memory_order_relaxed); }


// Heads per work item of the fused path: a divisor of the heads per group (an
// item's heads share B and C).  More heads per item share more of the item's
// set-up (Gram tiles, B^T and C fragments); fewer give more items.  The
// largest of 4, 2 that leaves at least two items per compute unit (measured
// best at the 2.7B layer shape), else the largest that leaves one, else 1;
// then a divisor up to 6 that fills whole rounds where that is clearly cheaper
// (below).  The heads_per_item tuning overrides it (ignored unless it divides
// the heads per group).

int64_t heads_per_workgroup(int64_t heads_per_group, int64_t items_per_head, int compute_units)
{
    if (const int64_t v = tuning(kTuneHeadsPerItem); v >= 1 && heads_per_group % v == 0) return v;
    // items_per_head: chunks x batch rows x groups, the items at one head per item
    int64_t hg = 1;
    bool found = false;
    for (int64_t need : {2, 1}) {
        for (int64_t h : {4, 2})
            if (heads_per_group % h == 0 && items_per_head * (heads_per_group / h) >= need * compute_units) {
                hg = h;
                found = true;
                break;
            }
        if (found) break;
    }
    // A divisor up to 6 replaces that choice when it is cheaper by rounds x
    // (heads per item + 1/2 of a head for the item's set-up) + 1/4 of a head
    // per head of an item (the longer an item, the longer a chunk's wait for
    // the chunk before it carries into its later heads).  At the 2.7B layer
    // shape 5 heads give 1,024 items (four rounds: 0.189 ms; 4 heads 0.188,
    // 10 heads 0.193, 20 heads 0.209); at the 130M layer shape 3 heads give 512
    // items (two rounds: 0.072 ms; 6 heads in one round 0.074-0.077).
    const auto cost = [&](int64_t h) {
        const int64_t items = items_per_head * (heads_per_group / h);
        return static_cast<double>((items + compute_units - 1) / compute_units) * (h + 0.5) + 0.25 * h;
    };
    double best = cost(hg);
    const double base = best;
    int64_t pick = hg;
    for (int64_t h = 1; h <= 6; ++h)
        if (heads_per_group % h == 0 && cost(h) < best) {
            best = cost(h);
            pick = h;
        }
    return best < base ? pick : hg;
}

WorkspaceLayout workspace_layout(int64_t b, int64_t H, int64_t P, int64_t N, int64_t G,
                                 int64_t Q, int64_t nC)
{
    WorkspaceLayout w;
    size_t off = kWorkspaceHeader;   // the status word sits in the header
    w.cs = off;
    off = align_up(off + sizeof(float) * static_cast<size_t>(b * H * nC * Q));
    w.info = off;
    off = align_up(off + sizeof(int4) * static_cast<size_t>(b * H * nC));
    w.gram = off;
    off = align_up(off + sizeof(float) * static_cast<size_t>(b * G * nC) * static_cast<size_t>(Q * Q));
    w.states = off;
    off = align_up(off + sizeof(float) * static_cast<size_t>(b * nC * H) * static_cast<size_t>(P * N));
    w.total = off;
    return w;
}

}  // namespace ssd

namespace {

// A packed row (seq_idx) runs through the fused kernels when it is one row of
// at most 2^31 - 1 tokens and nseq is valid.
bool fused_packed_ok(const ssd_problem* prob)
{
    return prob->batch == 1 && prob->nseq >= 1 && prob->nseq <= prob->seqlen && prob->seqlen <= INT32_MAX;
}

}  // namespace

extern "C" int ssd_workspace_bytes(const ssd_problem* prob, size_t* bytes)
{
    if (!bytes) return SSD_ERR_NULL_ARG;
    ssd::Shape s;
    const int rc = ssd::validate(prob, /*has_seq_idx=*/false, &s);  // size does not depend on it
    if (rc != SSD_OK) return rc;
    // The size of the path the forward will take: the fused kernels' layout
    // where they apply (a fraction of the general layout, which holds every
    // chunk state), else the general one.  Forcing the general path through
    // ssd_set_tuning changes the answer.
    const size_t general = ssd::workspace_layout(s.b, s.H, s.P, s.N, s.G, s.Q, s.nC).total;
    size_t need = general;
    if (ssd::tuning(ssd::kTuneForceGeneral) != 1 && ssd::fused_supported(s.P, s.N, s.Q, s.bf16)) {
        need = ssd::fused_layout(s.b, s.T, s.H, s.N, s.G, s.nC, 0).total;
        // a packed row of prob->nseq sequences (when seq_idx is passed) needs its chunk table
        if (fused_packed_ok(prob))
            need = std::max(need, ssd::fused_layout(1, s.T, s.H, s.N, s.G, s.nC, prob->nseq).total);
        else if (prob->batch == 1 && prob->nseq >= 1 && prob->nseq <= prob->seqlen)
            need = std::max(need, general);   // a packed row the fused kernels cannot index
    }
    *bytes = need;
    return SSD_OK;
}

extern "C" int ssd_block_workspace_bytes(const ssd_problem* prob, const ssd_block_opts* opts, size_t* bytes)
{
    if (!opts) return SSD_ERR_NULL_ARG;
    return ssd_workspace_bytes(prob, bytes);   // the block steps need no workspace of their own
}

namespace {

bool aligned16(const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; }

// Block options against the shape; fills the dt parameterisation.
int validate_block(const ssd_block_opts* o, const ssd::Shape& s, const void* y, ssd::DtTransform* dtx)
{
    if (!(o->dt_min >= 0.f) || !(o->dt_max >= o->dt_min)) return SSD_ERR_BAD_OPTION;   // NaN fails too
    if (!(o->norm_eps >= 0.f) || !std::isfinite(o->norm_eps)) return SSD_ERR_BAD_OPTION;
    const int64_t C = s.H * s.P;
    if (o->norm_group_size < 0 || (o->norm_group_size > 0 &&
                                   (o->norm_group_size % s.P != 0 || C % o->norm_group_size != 0)))
        return SSD_ERR_BAD_OPTION;
    if ((o->z || o->norm_group_size > 0) && (!aligned16(y) || (o->z && !aligned16(o->z)) ||
                                             (o->norm_weight && !aligned16(o->norm_weight))))
        return SSD_ERR_UNSUPPORTED_DIMS;
    dtx->bias = o->dt_bias;
    dtx->softplus = o->dt_softplus != 0;
    dtx->lo = o->dt_min;
    dtx->hi = o->dt_max;
    dtx->active = o->dt_bias || o->dt_softplus || o->dt_min > 0.f || o->dt_max < INFINITY;
    return SSD_OK;
}

int forward_impl(const ssd_problem* prob, const ssd_block_opts* opts, const void* x, const void* dt,
                 const float* A_log, const void* B, const void* C, const float* D,
                 const float* initial_states, const int32_t* seq_idx, void* y, float* final_states,
                 void* workspace, size_t workspace_bytes, void* stream, hipEvent_t ev_begin,
                 hipEvent_t ev_end, const ssd::SeqStartsArg* arg_starts = nullptr, int* status = nullptr,
                 bool reset_status = true, bool y32 = false)
{
    // y32 (the layer recomputed for the block gradients): y in float32, on the
    // fused kernels only (plain rows, chunk 256, no gate or normalisation)
    // arg_starts (a packed row by host offsets, instead of seq_idx): only on the
    // fused path, which the caller has checked; the workspace is its layout
    ssd::Shape s;
    int rc = ssd::validate(prob, seq_idx != nullptr || arg_starts != nullptr, &s);
    if (rc != SSD_OK) return rc;
    if (!x || !dt || !A_log || !B || !C || !y) return SSD_ERR_NULL_ARG;
    ssd::DtTransform dtx;
    if (opts && (rc = validate_block(opts, s, y, &dtx)) != SSD_OK) return rc;
    size_t need = 0;
    if (arg_starts)
        need = ssd::fused_layout(1, s.T, s.H, s.N, s.G, s.nC, s.nseq).total;
    else if (ssd_workspace_bytes(prob, &need) != SSD_OK)
        return SSD_ERR_WORKSPACE;
    if (!workspace || workspace_bytes < need) return SSD_ERR_WORKSPACE;
    // output side of the block: gate and grouped normalisation
    ssd::GateNormParams gn;
    gn.rows = s.b * s.T;
    gn.C = s.H * s.P;
    gn.group = opts ? opts->norm_group_size : 0;
    gn.y = y;
    gn.z = opts ? opts->z : nullptr;
    gn.weight = opts ? opts->norm_weight : nullptr;
    gn.eps = opts ? opts->norm_eps : 0.f;
    const bool post = gn.z || gn.group > 0;
    const bool force_unfused = ssd::tuning(ssd::kTuneForceGeneral) == 1;
    // status word: in the workspace's header unless the caller keeps it elsewhere
    if (!status) status = static_cast<int*>(workspace);
    if (arg_starts ||
        (!force_unfused && ssd::fused_supported(s.P, s.N, s.Q, s.bf16) && (!seq_idx || fused_packed_ok(prob)))) {
        const int64_t nseq = seq_idx || arg_starts ? s.nseq : 0;
        const ssd::FusedLayout fw = ssd::fused_layout(s.b, s.T, s.H, s.N, s.G, s.nC, nseq);
        ssd::FusedParams f;
        f.b = s.b;
        f.T = s.T;
        f.H = s.H;
        f.P = s.P;
        f.N = s.N;
        f.G = s.G;
        f.nC = fw.nC;
        int dev = 0, cus = 256;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
            return SSD_ERR_LAUNCH;
        f.HG = ssd::heads_per_workgroup(s.H / s.G, fw.nC * s.b * s.G, cus);
        // The chain of state passing takes about nC chunk steps one after the
        // other (a step: a chunk's wait, state load, combine and publish), the
        // work about rounds x heads per item head-times.  Where the chain is
        // the longer (few heads and batch rows, many chunks: nC >= 2 x rounds
        // x heads per item), each chunk publishes its state before its left
        // factor, which shortens every chain step by the left factor and the
        // output stage (the 2.7B layer split 8 ways by heads: 0.056 ms against
        // 0.081); elsewhere it sets the flag after the output stage, which
        // measures up to 2 % faster there.  The early_state_flag tuning
        // overrides it.
        // A packed row of several sequences, its chunks taken by their index
        // within their sequence (below), has a chain per sequence: about
        // table entries / sequences chunks long (the longest is unknown here
        // when the boundaries are on the device).
        const bool by_depth = nseq > 1 && ssd::tuning(ssd::kTunePackedOrder) != 1;
        const int64_t items = fw.nC * s.b * (s.H / f.HG);
        const int64_t rounds = (items + cus - 1) / cus;
        const int64_t chain = by_depth ? (fw.nC + nseq - 1) / nseq : fw.nC;
        f.early_flag = chain >= 2 * rounds * f.HG ? 1 : 0;
        if (const int64_t ef = ssd::tuning(ssd::kTuneEarlyFlag); ef == 1 || ef == 2) f.early_flag = ef == 2;
        // The right factor in the diagonal block's pass (x read from LDS once for
        // both; with N = 256 the first column block's) shortens a head's
        // matrix-product phase but holds more registers through it; measured
        // faster with long items and the late flag (2.7B layer 0.1864 ms against
        // 0.1908, the state-size sweep at N = 64 0.549 against 0.597, at N = 256
        // 1.256 against 1.295) and slower with items of 1-3 heads (130M layer,
        // the 8-way head and sequence splits: 2-4 %) and with the early flag.
        f.fuse_rf = !f.early_flag && f.HG >= 4 && !y32 ? 1 : 0;
        if (const int64_t fr = ssd::tuning(ssd::kTuneFusedRightFactor); fr == 1 || fr == 2)
            f.fuse_rf = fr == 2 && !f.early_flag && !y32;
        f.status = status;
        f.reset_status = reset_status ? 1 : 0;
        if (const int64_t sl = ssd::tuning(ssd::kTuneStateWaitLimit); sl >= 1) f.spin_limit = sl;
        f.max_workgroups = static_cast<int>(ssd::tuning(ssd::kTuneMaxWorkgroups));
        f.y32 = y32 ? 1 : 0;
        f.x = x;
        f.dt = dt;
        f.A_log = A_log;
        f.B = B;
        f.C = C;
        f.D = D;
        f.init = initial_states;
        f.y = y;
        f.fin = final_states;
        char* base = static_cast<char*>(workspace);
        f.gram = reinterpret_cast<uint16_t*>(base + fw.gram);
        f.BT = reinterpret_cast<uint16_t*>(base + fw.BT);
        f.ring = reinterpret_cast<float*>(base + fw.ring);
        f.flags = reinterpret_cast<int*>(base + fw.flags);
        f.ticket = reinterpret_cast<int*>(base + fw.ticket);
        f.ring_rows = fw.ring_rows;
        if (seq_idx || arg_starts) {
            f.seq_idx = seq_idx;
            f.arg_starts = arg_starts;
            f.nseq = nseq;
            f.starts = reinterpret_cast<int*>(base + fw.starts);
            f.vtab = reinterpret_cast<int4*>(base + fw.vtab);
            f.vcount = f.ticket + 2;
            // Several sequences: chunks taken by their index within their
            // sequence rather than in table order (k_seq_order), so that the
            // chunks in flight are mostly of different sequences.
            if (by_depth) f.vorder = reinterpret_cast<int*>(base + fw.vorder);
        }
        f.dtx = dtx;
        // The chunk kernel gates, and normalises one-head groups, in its output
        // stage.  Wider groups take one more pass, which then also gates (z is
        // read once either way, and gating in that pass measured faster than in
        // the chunk kernel).  The separate_block_post tuning leaves gate and
        // normalisation to that pass in every case.
        const bool separate = ssd::tuning(ssd::kTuneSeparatePost) == 1;
        if (post && !separate && (gn.group == 0 || gn.group == s.P)) {
            f.z = gn.z;
            if (gn.group == s.P) {
                f.norm_head = 1;
                f.norm_weight = gn.weight;
                f.norm_eps = gn.eps;
            }
            gn.z = nullptr;
            gn.group = 0;
        }
        hipError_t err = ssd::launch_fused(f, static_cast<hipStream_t>(stream), ev_begin, ev_end);
        if (err == hipSuccess && (gn.z || gn.group > 0))
            err = ssd::launch_gate_norm(gn, s.bf16, static_cast<hipStream_t>(stream));
        return err == hipSuccess ? SSD_OK : SSD_ERR_LAUNCH;
    }
    if (y32) return SSD_ERR_UNSUPPORTED_DIMS;   // float32 y only from the fused kernels
    const ssd::WorkspaceLayout w = ssd::workspace_layout(s.b, s.H, s.P, s.N, s.G, s.Q, s.nC);

    ssd::Params p;
    p.b = s.b;
    p.T = s.T;
    p.H = s.H;
    p.P = s.P;
    p.N = s.N;
    p.G = s.G;
    p.Q = s.Q;
    p.nC = s.nC;
    p.nseq = s.nseq;
    p.x = x;
    p.dt = dt;
    p.A_log = A_log;
    p.B = B;
    p.C = C;
    p.D = D;
    p.init = initial_states;
    p.seq_idx = seq_idx;
    p.y = y;
    p.fin = final_states;
    char* ws = static_cast<char*>(workspace);
    p.cs = reinterpret_cast<float*>(ws + w.cs);
    p.info = reinterpret_cast<int4*>(ws + w.info);
    p.gram = reinterpret_cast<float*>(ws + w.gram);
    p.states = reinterpret_cast<float*>(ws + w.states);
    p.dtx = dtx;
    p.status = reset_status ? status : nullptr;
    hipError_t err = ssd::launch_unfused(p, s.bf16, static_cast<hipStream_t>(stream), ev_begin, ev_end);
    if (err == hipSuccess && post) err = ssd::launch_gate_norm(gn, s.bf16, static_cast<hipStream_t>(stream));
    return err == hipSuccess ? SSD_OK : SSD_ERR_LAUNCH;
}

}  // namespace

extern "C" int ssd_forward(const ssd_problem* prob, const void* x, const void* dt,
                           const float* A_log, const void* B, const void* C, const float* D,
                           const float* initial_states, const int32_t* seq_idx, void* y,
                           float* final_states, void* workspace, size_t workspace_bytes,
                           void* stream)
{
    return forward_impl(prob, nullptr, x, dt, A_log, B, C, D, initial_states, seq_idx, y, final_states,
                        workspace, workspace_bytes, stream, nullptr, nullptr);
}

extern "C" int ssd_forward_timed(const ssd_problem* prob, const void* x, const void* dt,
                                 const float* A_log, const void* B, const void* C,
                                 const float* D, const float* initial_states,
                                 const int32_t* seq_idx, void* y, float* final_states,
                                 void* workspace, size_t workspace_bytes, void* stream,
                                 void* event_begin, void* event_end)
{
    return forward_impl(prob, nullptr, x, dt, A_log, B, C, D, initial_states, seq_idx, y, final_states,
                        workspace, workspace_bytes, stream, static_cast<hipEvent_t>(event_begin),
                        static_cast<hipEvent_t>(event_end));
}

extern "C" int ssd_forward_block(const ssd_problem* prob, const ssd_block_opts* opts, const void* x,
                                 const void* dt, const float* A_log, const void* B, const void* C,
                                 const float* D, const float* initial_states, const int32_t* seq_idx,
                                 void* y, float* final_states, void* workspace, size_t workspace_bytes,
                                 void* stream)
{
    if (!opts) return SSD_ERR_NULL_ARG;
    return forward_impl(prob, opts, x, dt, A_log, B, C, D, initial_states, seq_idx, y, final_states,
                        workspace, workspace_bytes, stream, nullptr, nullptr);
}

extern "C" int ssd_forward_block_timed(const ssd_problem* prob, const ssd_block_opts* opts, const void* x,
                                       const void* dt, const float* A_log, const void* B, const void* C,
                                       const float* D, const float* initial_states, const int32_t* seq_idx,
                                       void* y, float* final_states, void* workspace, size_t workspace_bytes,
                                       void* stream, void* event_begin, void* event_end)
{
    if (!opts) return SSD_ERR_NULL_ARG;
    return forward_impl(prob, opts, x, dt, A_log, B, C, D, initial_states, seq_idx, y, final_states,
                        workspace, workspace_bytes, stream, static_cast<hipEvent_t>(event_begin),
                        static_cast<hipEvent_t>(event_end));
}

extern "C" int ssd_decode_step(const ssd_problem* prob, const void* x, const void* dt,
                               const float* A_log, const void* B, const void* C, const float* D,
                               float* state, void* y, void* stream)
{
    if (!prob) return SSD_ERR_NULL_ARG;
    if (prob->dtype != SSD_DTYPE_F32 && prob->dtype != SSD_DTYPE_BF16) return SSD_ERR_BAD_DTYPE;
    if (prob->batch < 1 || prob->nheads < 1 || prob->headdim < 1 || prob->dstate < 1 ||
        prob->ngroups < 1 || prob->nheads % prob->ngroups != 0)
        return SSD_ERR_BAD_SHAPE;
    if (prob->headdim % 16 != 0 || prob->headdim > 128 || prob->dstate % 16 != 0 ||
        prob->dstate > 256 || reinterpret_cast<uintptr_t>(state) % 16 != 0)
        return SSD_ERR_UNSUPPORTED_DIMS;
    if (!x || !dt || !A_log || !B || !C || !state || !y) return SSD_ERR_NULL_ARG;
    if (prob->batch > 65535 || prob->nheads > 65535 ||
        static_cast<double>(prob->batch) * prob->nheads * prob->headdim * prob->dstate > 16.0 * ssd::kMaxElemsPublic)
        return SSD_ERR_TOO_LARGE;
    ssd::DecodeParams p;
    p.b = prob->batch;
    p.H = prob->nheads;
    p.P = prob->headdim;
    p.N = prob->dstate;
    p.G = prob->ngroups;
    p.x = x;
    p.dt = dt;
    p.A_log = A_log;
    p.B = B;
    p.C = C;
    p.D = D;
    p.state = state;
    p.y = y;
    const hipError_t err =
        ssd::launch_decode(p, prob->dtype == SSD_DTYPE_BF16, static_cast<hipStream_t>(stream));
    return err == hipSuccess ? SSD_OK : SSD_ERR_LAUNCH;
}

namespace {

// Shape checks of the span entry points: those of ssd_forward, without the
// chunk size (spans use their own tiling) and without packed rows.
int validate_span(const ssd_problem* prob)
{
    if (!prob) return SSD_ERR_NULL_ARG;
    ssd_problem q = *prob;
    q.chunk_size = 256;
    ssd::Shape s;
    return ssd::validate(&q, false, &s);
}

}  // namespace

extern "C" int ssd_span_decay(const ssd_problem* prob, const void* dt, const float* A_log, float* decay,
                              void* stream)
{
    const int rc = validate_span(prob);
    if (rc != SSD_OK) return rc;
    if (!dt || !A_log || !decay) return SSD_ERR_NULL_ARG;
    const hipError_t err = ssd::launch_span_decay(prob->batch, prob->seqlen, prob->nheads, dt, A_log, decay,
                                                  prob->dtype == SSD_DTYPE_BF16, static_cast<hipStream_t>(stream));
    return err == hipSuccess ? SSD_OK : SSD_ERR_LAUNCH;
}

extern "C" int ssd_span_combine(int64_t nspans, const ssd_problem* prob, const float* decay,
                                const float* local_final, const float* initial_states, float* entering,
                                float* final_states, void* stream)
{
    const int rc = validate_span(prob);
    if (rc != SSD_OK) return rc;
    if (nspans < 1 || nspans > 65536) return SSD_ERR_BAD_SHAPE;
    if (!decay || !local_final || !entering) return SSD_ERR_NULL_ARG;
    const auto a16 = [](const void* q) { return reinterpret_cast<uintptr_t>(q) % 16 == 0; };
    if (!a16(local_final) || !a16(entering) || !a16(initial_states) || !a16(final_states))
        return SSD_ERR_UNSUPPORTED_DIMS;
    const int64_t PN = prob->headdim * prob->dstate;
    if (static_cast<double>(nspans) * prob->batch * prob->nheads * PN > 16.0 * ssd::kMaxElemsPublic)
        return SSD_ERR_TOO_LARGE;
    const hipError_t err = ssd::launch_span_combine(nspans, prob->batch * prob->nheads, PN, decay, local_final,
                                                    initial_states, entering, final_states,
                                                    static_cast<hipStream_t>(stream));
    return err == hipSuccess ? SSD_OK : SSD_ERR_LAUNCH;
}

extern "C" int ssd_span_correct_workspace_bytes(const ssd_problem* prob, size_t* bytes)
{
    if (!bytes) return SSD_ERR_NULL_ARG;
    const int rc = validate_span(prob);
    if (rc != SSD_OK) return rc;
    *bytes = sizeof(float) * static_cast<size_t>(prob->batch * prob->nheads * ssd::span_chunks(prob->seqlen));
    return SSD_OK;
}

extern "C" int ssd_span_correct(const ssd_problem* prob, const void* dt, const float* A_log, const void* C,
                                const float* entering, void* y, void* workspace, size_t workspace_bytes,
                                void* stream)
{
    size_t need = 0;
    const int rc = ssd_span_correct_workspace_bytes(prob, &need);
    if (rc != SSD_OK) return rc;
    if (!dt || !A_log || !C || !entering || !y) return SSD_ERR_NULL_ARG;
    const auto a16 = [](const void* q) { return reinterpret_cast<uintptr_t>(q) % 16 == 0; };
    if (!a16(C) || !a16(entering) || !a16(y)) return SSD_ERR_UNSUPPORTED_DIMS;   // 16-byte vectors
    if (!workspace || workspace_bytes < need) return SSD_ERR_WORKSPACE;
    ssd::SpanParams p;
    p.b = prob->batch;
    p.T = prob->seqlen;
    p.H = prob->nheads;
    p.P = prob->headdim;
    p.N = prob->dstate;
    p.G = prob->ngroups;
    p.nC = ssd::span_chunks(prob->seqlen);
    p.dt = dt;
    p.A_log = A_log;
    p.C = C;
    p.entering = entering;
    p.y = y;
    p.sums = static_cast<float*>(workspace);
    const hipError_t err =
        ssd::launch_span_correct(p, prob->dtype == SSD_DTYPE_BF16, static_cast<hipStream_t>(stream));
    return err == hipSuccess ? SSD_OK : SSD_ERR_LAUNCH;
}

namespace {

// Shape checks of the backward: those of ssd_forward without packed rows; the
// chunk size is not used (the backward has its own decomposition).
// The matrix-core path where it applies; the force_general_path tuning (as
// for the forward) forces the general one.
bool backward_fast(const ssd::Shape& s)
{
    if (ssd::tuning(ssd::kTuneForceGeneral) == 1) return false;
    return ssd::bwd_fast_supported(s.bf16, s.P, s.N);
}

int backward_plan(const ssd_problem* prob, ssd::BwdParams* p, ssd::BwdLayout* l, bool* fast)
{
    if (!prob) return SSD_ERR_NULL_ARG;
    ssd_problem q = *prob;
    q.chunk_size = 256;
    ssd::Shape s;
    const int rc = ssd::validate(&q, false, &s);
    if (rc != SSD_OK) return rc;
    *fast = backward_fast(s);
    const int64_t Q = *fast ? ssd::kBwdQFast : ssd::kBwdQ;
    p->b = s.b;
    p->T = s.T;
    p->H = s.H;
    p->P = s.P;
    p->N = s.N;
    p->G = s.G;
    p->nC = (s.T + Q - 1) / Q;
    if (static_cast<double>(p->b) * p->nC * p->H * p->P * p->N > 16.0 * ssd::kMaxElemsPublic)
        return SSD_ERR_TOO_LARGE;
    ssd::bwd_slices(p->b, p->nC, p->G, p->H / p->G, &p->S, &p->hs);
    if (const int64_t v = ssd::tuning(ssd::kTuneBwdHeadsPerSlice); v >= 1) {
        p->hs = v < p->H / p->G ? v : p->H / p->G;
        p->S = (p->H / p->G + p->hs - 1) / p->hs;
    }
    *l = ssd::bwd_layout(p->b, p->T, p->H, p->P, p->N, p->G, p->nC, p->S, *fast);
    return SSD_OK;
}

int backward_impl(const ssd_problem* prob, const void* x, const void* dt, const float* A_log, const void* B,
                  const void* C, const float* D, const float* initial_states, const void* dy,
                  const float* dfinal_states, void* dx, void* ddt, float* dA_log, void* dB, void* dC, float* dD,
                  float* dinitial_states, void* workspace, size_t workspace_bytes, void* stream,
                  void* ev_begin, void* ev_end, bool h32 = false)
{
    // h32 (the block gradients): dt, dy float32 in, ddt float32 out, on the
    // matrix-core path only
    ssd::BwdParams p{};
    ssd::BwdLayout l{};
    bool fast = false;
    const int rc = backward_plan(prob, &p, &l, &fast);
    if (rc != SSD_OK) return rc;
    if (h32 && !fast) return SSD_ERR_UNSUPPORTED_DIMS;
    p.h32 = h32 ? 1 : 0;
    if (!x || !dt || !A_log || !B || !C || !dy || !dx || !ddt || !dA_log || !dB || !dC)
        return SSD_ERR_NULL_ARG;
    if (!aligned16(initial_states) || !aligned16(dfinal_states) || !aligned16(dinitial_states) ||
        !aligned16(x) || !aligned16(B) || !aligned16(C) || !aligned16(dy) || !aligned16(dx))
        return SSD_ERR_UNSUPPORTED_DIMS;   // read and written as 16-byte vectors
    if (!workspace || workspace_bytes < l.total) return SSD_ERR_WORKSPACE;
    char* ws = static_cast<char*>(workspace);
    p.x = x;
    p.dt = dt;
    p.A_log = A_log;
    p.B = B;
    p.C = C;
    p.D = D;
    p.init = initial_states;
    p.dy = dy;
    p.dfinal = dfinal_states;
    p.dx = dx;
    p.ddt = ddt;
    p.dA_log = dA_log;
    p.dB = dB;
    p.dC = dC;
    p.dD = D ? dD : nullptr;
    p.dinit = dinitial_states;
    p.cs = fast ? nullptr : reinterpret_cast<float*>(ws + l.cs);
    p.hin = reinterpret_cast<float*>(ws + l.hin);
    p.gn = fast ? nullptr : reinterpret_cast<float*>(ws + l.gn);
    p.gnT = fast ? reinterpret_cast<float*>(ws + l.gnT) : nullptr;
    p.dBp = reinterpret_cast<float*>(ws + l.dBp);
    p.dCp = reinterpret_cast<float*>(ws + l.dCp);
    p.dAp = reinterpret_cast<float*>(ws + l.dAp);
    p.dDp = reinterpret_cast<float*>(ws + l.dDp);
    const hipStream_t st = static_cast<hipStream_t>(stream);
    const hipEvent_t e0 = static_cast<hipEvent_t>(ev_begin), e1 = static_cast<hipEvent_t>(ev_end);
    const hipError_t err = fast ? ssd::launch_backward_fast(p, st, e0, e1)
                                : ssd::launch_backward(p, prob->dtype == SSD_DTYPE_BF16, st, e0, e1);
    return err == hipSuccess ? SSD_OK : SSD_ERR_LAUNCH;
}

}  // namespace

extern "C" int ssd_backward_workspace_bytes(const ssd_problem* prob, size_t* bytes)
{
    if (!bytes) return SSD_ERR_NULL_ARG;
    ssd::BwdParams p{};
    ssd::BwdLayout l{};
    bool fast = false;
    const int rc = backward_plan(prob, &p, &l, &fast);
    if (rc != SSD_OK) return rc;
    *bytes = l.total;
    return SSD_OK;
}

extern "C" int ssd_backward(const ssd_problem* prob, const void* x, const void* dt, const float* A_log,
                            const void* B, const void* C, const float* D, const float* initial_states,
                            const void* dy, const float* dfinal_states, void* dx, void* ddt, float* dA_log,
                            void* dB, void* dC, float* dD, float* dinitial_states, void* workspace,
                            size_t workspace_bytes, void* stream)
{
    return backward_impl(prob, x, dt, A_log, B, C, D, initial_states, dy, dfinal_states, dx, ddt, dA_log, dB, dC,
                         dD, dinitial_states, workspace, workspace_bytes, stream, nullptr, nullptr);
}

extern "C" int ssd_backward_timed(const ssd_problem* prob, const void* x, const void* dt, const float* A_log,
                                  const void* B, const void* C, const float* D, const float* initial_states,
                                  const void* dy, const float* dfinal_states, void* dx, void* ddt,
                                  float* dA_log, void* dB, void* dC, float* dD, float* dinitial_states,
                                  void* workspace, size_t workspace_bytes, void* stream, void* event_begin,
                                  void* event_end)
{
    return backward_impl(prob, x, dt, A_log, B, C, D, initial_states, dy, dfinal_states, dx, ddt, dA_log, dB, dC,
                         dD, dinitial_states, workspace, workspace_bytes, stream, event_begin, event_end);
}

namespace {

// Workspace of the block backward: the dt step's output, the layer's output
// (recomputed), its gradient, the layer's dt gradient -- all four float32 --
// the normalisation's 1 / r per (row, group), the row-chunk partials of
// d weight and d bias, and one region shared by the forward and the layer
// backward (they run one after the other).
//
// Three ways to run it:
//   kF32      float32 activations: every kernel in float32;
//   kMatrix   bf16 activations at the matrix-core shapes (headdim 64, dstate
//             64 or 128): the layer recomputed by the fused kernels with y in
//             float32, the layer backward on the matrix cores with float32
//             dt, dy and ddt;
//   kWidened  bf16 activations at any other shape: the activations widened to
//             float32 (exactly), the call run as kF32 on the copies, and the
//             activation-dtype gradients rounded back to bf16.
enum BlockMode { kF32, kMatrix, kWidened };

struct BlockBwdLayout {
    BlockMode mode;
    size_t dt, y, dy, ddt, inv_rms, dw_part, db_part, shared, total;
    // kWidened: float32 copies of the inputs and float32 gradients, then the
    // float32 call's own workspace at `inner`
    size_t wx, wdt, wB, wC, wdout, wz, gx, gdt, gB, gC, gz, inner;
};

BlockMode block_mode(const ssd::Shape& s)
{
    if (!s.bf16) return kF32;
    if (ssd::tuning(ssd::kTuneForceGeneral) != 1 && ssd::fused_supported(s.P, s.N, 256, true) &&
        ssd::bwd_fast_supported(true, s.P, s.N))
        return kMatrix;
    return kWidened;
}

int block_backward_plan(const ssd_problem* prob, const ssd_block_opts* opts, BlockBwdLayout* l)
{
    if (!prob || !opts) return SSD_ERR_NULL_ARG;
    ssd::Shape s;
    int rc = ssd::validate(prob, false, &s);
    if (rc != SSD_OK) return rc;
    l->mode = block_mode(s);
    size_t off = ssd::kWorkspaceHeader;   // the recomputed forward's status word sits in the header
    const auto take = [&](size_t bytes) {
        const size_t o = off;
        off += ssd::align_up(bytes);
        return o;
    };
    const size_t rows = static_cast<size_t>(prob->batch * prob->seqlen);
    const size_t H = static_cast<size_t>(prob->nheads), Cc = H * static_cast<size_t>(prob->headdim);
    if (l->mode == kWidened) {
        const size_t GN = static_cast<size_t>(prob->ngroups * prob->dstate);
        l->wx = take(rows * Cc * 4);
        l->wdt = take(rows * H * 4);
        l->wB = take(rows * GN * 4);
        l->wC = take(rows * GN * 4);
        l->wdout = take(rows * Cc * 4);
        l->wz = take(opts->z ? rows * Cc * 4 : 0);
        l->gx = take(rows * Cc * 4);
        l->gdt = take(rows * H * 4);
        l->gB = take(rows * GN * 4);
        l->gC = take(rows * GN * 4);
        l->gz = take(opts->z ? rows * Cc * 4 : 0);
        ssd_problem q = *prob;
        q.dtype = SSD_DTYPE_F32;
        BlockBwdLayout inner{};
        if ((rc = block_backward_plan(&q, opts, &inner)) != SSD_OK) return rc;
        l->inner = take(inner.total);
        l->total = off;
        return SSD_OK;
    }
    size_t fwd = 0, bwd = 0;
    ssd_problem qf = *prob;
    if (l->mode == kMatrix) qf.chunk_size = 256;   // the fused kernels' chunk (the result does not depend on it)
    if ((rc = ssd_workspace_bytes(&qf, &fwd)) != SSD_OK) return rc;
    if ((rc = ssd_backward_workspace_bytes(prob, &bwd)) != SSD_OK) return rc;
    const size_t nch = static_cast<size_t>(ssd::block_bwd_row_chunks(static_cast<int64_t>(rows)));
    if (nch > 65535) return SSD_ERR_TOO_LARGE;   // row chunks on grid y
    const size_t groups = opts->norm_group_size > 0 ? Cc / static_cast<size_t>(opts->norm_group_size) : 0;
    l->dt = take(rows * H * 4);
    l->y = take(rows * Cc * 4);
    l->dy = take(rows * Cc * 4);
    l->ddt = take(rows * H * 4);
    l->inv_rms = take(rows * groups * 4);
    l->dw_part = take(opts->norm_weight && groups ? nch * Cc * 4 : 0);
    l->db_part = take(opts->dt_bias ? nch * H * 4 : 0);
    l->shared = take(fwd > bwd ? fwd : bwd);
    l->total = off;
    return SSD_OK;
}

// The block backward on validated arguments (kF32 or kMatrix); `status` is
// where the recomputed forward leaves its status word.
int block_backward_run(const ssd_problem* prob, const ssd_block_opts* opts, const BlockBwdLayout& l,
                       const ssd::Shape& s, const void* x, const void* dt, const float* A_log, const void* B,
                       const void* C, const float* D, const float* initial_states, const void* dout,
                       const float* dfinal_states, void* dx, void* ddt, float* dA_log, void* dB, void* dC,
                       float* dD, float* dinitial_states, float* ddt_bias, void* dz, float* dnorm_weight, char* ws,
                       int* status, void* stream)
{
    const bool bf16 = s.bf16;
    const bool matrix = l.mode == kMatrix;
    const hipStream_t st = static_cast<hipStream_t>(stream);
    const size_t shared_bytes = l.total - l.shared;

    ssd::BlockBwdParams p{};
    p.rows = s.b * s.T;
    p.H = s.H;
    p.C = s.H * s.P;
    p.group = opts->norm_group_size;
    p.dt_raw = dt;
    p.bias = opts->dt_bias;
    p.softplus = opts->dt_softplus != 0;
    p.lo = opts->dt_min;
    p.hi = opts->dt_max;
    p.dt = ws + l.dt;
    p.ddt = ws + l.ddt;
    p.ddt_raw = ddt;
    p.dbias_part = opts->dt_bias ? reinterpret_cast<float*>(ws + l.db_part) : nullptr;
    p.ddt_bias = opts->dt_bias ? ddt_bias : nullptr;
    p.y = ws + l.y;
    p.z = opts->z;
    p.w = opts->norm_group_size > 0 ? opts->norm_weight : nullptr;
    p.eps = opts->norm_eps;
    p.dout = dout;
    p.dy = ws + l.dy;
    p.dz = dz;
    p.inv_rms = opts->norm_group_size > 0 ? reinterpret_cast<float*>(ws + l.inv_rms) : nullptr;
    p.dw_part = reinterpret_cast<float*>(ws + l.dw_part);
    p.dw = p.w ? dnorm_weight : nullptr;

    // 1. the dt step (float32); 2. the layer's output, recomputed in float32:
    // with bf16 activations the fused kernels apply the dt step themselves, to
    // the raw dt, exactly as the block forward does
    if (ssd::launch_block_dt_apply(p, bf16, st) != hipSuccess) return SSD_ERR_LAUNCH;
    int rc;
    if (matrix) {
        ssd_problem q = *prob;
        q.chunk_size = 256;
        ssd_block_opts dto = *opts;   // the dt step only
        dto.z = nullptr;
        dto.norm_weight = nullptr;
        dto.norm_group_size = 0;
        rc = forward_impl(&q, &dto, x, dt, A_log, B, C, D, initial_states, nullptr, ws + l.y, nullptr,
                          ws + l.shared, shared_bytes, stream, nullptr, nullptr, nullptr, status, true,
                          /*y32=*/true);
    } else {
        rc = forward_impl(prob, nullptr, x, p.dt, A_log, B, C, D, initial_states, nullptr, ws + l.y, nullptr,
                          ws + l.shared, shared_bytes, stream, nullptr, nullptr, nullptr, status);
    }
    if (rc != SSD_OK) return rc == SSD_ERR_LAUNCH ? rc : SSD_ERR_LAUNCH;
    // 3. gate and normalisation: dy (the block's output gradient when neither is on)
    const bool post = opts->z || opts->norm_group_size > 0;
    const void* dy = dout;
    if (post) {
        if (ssd::launch_block_out_bwd(p, bf16, st) != hipSuccess) return SSD_ERR_LAUNCH;
        dy = p.dy;
    } else if (matrix) {   // the layer takes dy in float32
        if (ssd::launch_widen(dout, reinterpret_cast<float*>(p.dy), p.rows * p.C, st) != hipSuccess)
            return SSD_ERR_LAUNCH;
        dy = p.dy;
    }
    // 4. the layer
    rc = backward_impl(prob, x, p.dt, A_log, B, C, D, initial_states, dy, dfinal_states, dx, ws + l.ddt, dA_log,
                       dB, dC, dD, dinitial_states, ws + l.shared, shared_bytes, stream, nullptr, nullptr,
                       /*h32=*/matrix);
    if (rc != SSD_OK) return rc == SSD_ERR_LAUNCH ? rc : SSD_ERR_LAUNCH;
    // 5. the dt step
    return ssd::launch_block_dt_bwd(p, bf16, st) == hipSuccess ? SSD_OK : SSD_ERR_LAUNCH;
}

}  // namespace

extern "C" int ssd_backward_block_workspace_bytes(const ssd_problem* prob, const ssd_block_opts* opts,
                                                  size_t* bytes)
{
    if (!bytes) return SSD_ERR_NULL_ARG;
    BlockBwdLayout l{};
    const int rc = block_backward_plan(prob, opts, &l);
    if (rc != SSD_OK) return rc;
    *bytes = l.total;
    return SSD_OK;
}

extern "C" int ssd_backward_block(const ssd_problem* prob, const ssd_block_opts* opts, const void* x,
                                  const void* dt, const float* A_log, const void* B, const void* C,
                                  const float* D, const float* initial_states, const void* dout,
                                  const float* dfinal_states, void* dx, void* ddt, float* dA_log, void* dB,
                                  void* dC, float* dD, float* dinitial_states, float* ddt_bias, void* dz,
                                  float* dnorm_weight, void* workspace, size_t workspace_bytes, void* stream)
{
    BlockBwdLayout l{};
    int rc = block_backward_plan(prob, opts, &l);
    if (rc != SSD_OK) return rc;
    ssd::Shape s;
    if ((rc = ssd::validate(prob, false, &s)) != SSD_OK) return rc;
    ssd::DtTransform dtx;
    if ((rc = validate_block(opts, s, dout, &dtx)) != SSD_OK) return rc;
    if (!x || !dt || !A_log || !B || !C || !dout || !dx || !ddt || !dA_log || !dB || !dC) return SSD_ERR_NULL_ARG;
    if (opts->z && !dz) return SSD_ERR_NULL_ARG;
    // every check of the steps below is made here, before any work is enqueued
    if (!aligned16(x) || !aligned16(B) || !aligned16(C) || !aligned16(dx) || !aligned16(dout) ||
        (dz && !aligned16(dz)) || !aligned16(initial_states) || !aligned16(dfinal_states) ||
        !aligned16(dinitial_states))
        return SSD_ERR_UNSUPPORTED_DIMS;
    if (!workspace || workspace_bytes < l.total) return SSD_ERR_WORKSPACE;
    char* ws = static_cast<char*>(workspace);
    int* status = reinterpret_cast<int*>(ws);
    if (l.mode != kWidened)
        return block_backward_run(prob, opts, l, s, x, dt, A_log, B, C, D, initial_states, dout, dfinal_states, dx,
                                  ddt, dA_log, dB, dC, dD, dinitial_states, ddt_bias, dz, dnorm_weight, ws, status,
                                  stream);
    // bf16 activations outside the matrix-core shapes: the float32 call on
    // widened copies, its activation-dtype gradients rounded back to bf16
    const hipStream_t st = static_cast<hipStream_t>(stream);
    const int64_t rows = s.b * s.T, HP = s.H * s.P, GN = s.G * s.N;
    float* wx = reinterpret_cast<float*>(ws + l.wx);
    float* wdt = reinterpret_cast<float*>(ws + l.wdt);
    float* wB = reinterpret_cast<float*>(ws + l.wB);
    float* wC = reinterpret_cast<float*>(ws + l.wC);
    float* wdout = reinterpret_cast<float*>(ws + l.wdout);
    float* wz = opts->z ? reinterpret_cast<float*>(ws + l.wz) : nullptr;
    if (ssd::launch_widen(x, wx, rows * HP, st) != hipSuccess || ssd::launch_widen(dt, wdt, rows * s.H, st) != hipSuccess ||
        ssd::launch_widen(B, wB, rows * GN, st) != hipSuccess || ssd::launch_widen(C, wC, rows * GN, st) != hipSuccess ||
        ssd::launch_widen(dout, wdout, rows * HP, st) != hipSuccess ||
        (wz && ssd::launch_widen(opts->z, wz, rows * HP, st) != hipSuccess))
        return SSD_ERR_LAUNCH;
    ssd_problem q = *prob;
    q.dtype = SSD_DTYPE_F32;
    ssd_block_opts o32 = *opts;
    o32.z = wz;
    BlockBwdLayout inner{};
    ssd::Shape s32;
    if (block_backward_plan(&q, &o32, &inner) != SSD_OK || ssd::validate(&q, false, &s32) != SSD_OK)
        return SSD_ERR_LAUNCH;   // cannot happen: the same shape validated above
    float* gx = reinterpret_cast<float*>(ws + l.gx);
    float* gdt = reinterpret_cast<float*>(ws + l.gdt);
    float* gB = reinterpret_cast<float*>(ws + l.gB);
    float* gC = reinterpret_cast<float*>(ws + l.gC);
    float* gz = wz ? reinterpret_cast<float*>(ws + l.gz) : nullptr;
    rc = block_backward_run(&q, &o32, inner, s32, wx, wdt, A_log, wB, wC, D, initial_states, wdout, dfinal_states,
                            gx, gdt, dA_log, gB, gC, dD, dinitial_states, ddt_bias, gz, dnorm_weight, ws + l.inner,
                            status, stream);
    if (rc != SSD_OK) return rc;
    if (ssd::launch_narrow(gx, dx, rows * HP, st) != hipSuccess || ssd::launch_narrow(gdt, ddt, rows * s.H, st) != hipSuccess ||
        ssd::launch_narrow(gB, dB, rows * GN, st) != hipSuccess || ssd::launch_narrow(gC, dC, rows * GN, st) != hipSuccess ||
        (gz && ssd::launch_narrow(gz, dz, rows * HP, st) != hipSuccess))
        return SSD_ERR_LAUNCH;
    return SSD_OK;
}

namespace {

// Packed rows: the sequences are independent, so the backward runs on each
// sequence's token range as a problem of its own (pointer slices of the
// packed tensors; one state per sequence), and the per-sequence dA_log and dD
// are summed at the end.  seq_starts (host): nseq + 1 offsets, 0 = first <
// ... < last = seqlen.
// Packed-row backward in one launch (matrix-core path): every sequence cut
// into 64-token chunks of its own from a chunk table built on the device from
// the offsets handed over by value; b = 1 and nC = the table's capacity.
struct PackedBwdLayout {
    ssd::BwdLayout l;
    size_t starts, vtab, seq_first, vcount, total;
};

bool packed_backward_ok(const ssd_problem* prob)
{
    if (ssd::tuning(ssd::kTuneVarlenPerSequence) == 1 || ssd::tuning(ssd::kTuneForceGeneral) == 1) return false;
    ssd_problem q = *prob;
    q.chunk_size = 256;
    ssd::Shape s;
    if (ssd::validate(&q, true, &s) != SSD_OK) return false;
    return backward_fast(s) && prob->batch == 1 && prob->nseq <= ssd::kArgSeqs && prob->seqlen <= INT32_MAX;
}

int packed_backward_plan(const ssd_problem* prob, ssd::BwdParams* p, PackedBwdLayout* pl)
{
    ssd_problem q = *prob;
    q.chunk_size = 256;
    ssd::Shape s;
    const int rc = ssd::validate(&q, true, &s);
    if (rc != SSD_OK) return rc;
    const int64_t Q = ssd::kBwdQFast;
    p->b = 1;
    p->T = s.T;
    p->H = s.H;
    p->P = s.P;
    p->N = s.N;
    p->G = s.G;
    p->nseq = s.nseq;
    const int64_t nCd = (s.T + Q - 1) / Q;
    p->nC = std::min(nCd + s.nseq - 1, s.T);   // at most this many per-sequence chunks
    if (static_cast<double>(p->nC) * p->H * p->P * p->N > 16.0 * ssd::kMaxElemsPublic) return SSD_ERR_TOO_LARGE;
    ssd::bwd_slices(1, p->nC, p->G, p->H / p->G, &p->S, &p->hs);
    pl->l = ssd::bwd_layout(1, p->T, p->H, p->P, p->N, p->G, p->nC, p->S, true);
    size_t off = pl->l.total;
    pl->starts = off;
    off = ssd::align_up(off + sizeof(int) * static_cast<size_t>(s.nseq + 1));
    pl->vtab = off;
    off = ssd::align_up(off + sizeof(int4) * static_cast<size_t>(p->nC));
    pl->seq_first = off;
    off = ssd::align_up(off + sizeof(int) * static_cast<size_t>(s.nseq + 1));
    pl->vcount = off;
    off = ssd::align_up(off + sizeof(int));
    pl->total = off;
    return SSD_OK;
}

int varlen_plan(const ssd_problem* prob, const int64_t* seq_starts, size_t* sub_bytes, size_t* total)
{
    if (!prob || !seq_starts) return SSD_ERR_NULL_ARG;
    if (prob->batch != 1) return SSD_ERR_SEQIDX_BATCH;
    if (prob->nseq < 1 || prob->nseq > prob->seqlen) return SSD_ERR_BAD_SHAPE;
    if (seq_starts[0] != 0 || seq_starts[prob->nseq] != prob->seqlen) return SSD_ERR_BAD_SHAPE;
    for (int64_t s = 0; s < prob->nseq; ++s)
        if (seq_starts[s + 1] <= seq_starts[s]) return SSD_ERR_BAD_SHAPE;
    if (packed_backward_ok(prob)) {
        ssd::BwdParams p{};
        PackedBwdLayout pl{};
        const int rc = packed_backward_plan(prob, &p, &pl);
        if (rc != SSD_OK) return rc;
        *sub_bytes = 0;
        *total = pl.total;
        return SSD_OK;
    }
    size_t need = 0;
    for (int64_t s = 0; s < prob->nseq; ++s) {
        ssd_problem q = *prob;
        q.seqlen = seq_starts[s + 1] - seq_starts[s];
        size_t b = 0;
        const int rc = ssd_backward_workspace_bytes(&q, &b);
        if (rc != SSD_OK) return rc;
        if (b > need) need = b;
    }
    *sub_bytes = need;
    *total = ssd::align_up(2 * sizeof(float) * static_cast<size_t>(prob->nseq * prob->nheads)) + need;
    return SSD_OK;
}

}  // namespace

extern "C" int ssd_backward_varlen_workspace_bytes(const ssd_problem* prob, const int64_t* seq_starts,
                                                   size_t* bytes)
{
    if (!bytes) return SSD_ERR_NULL_ARG;
    size_t sub = 0;
    return varlen_plan(prob, seq_starts, &sub, bytes);
}

extern "C" int ssd_backward_varlen(const ssd_problem* prob, const int64_t* seq_starts, const void* x,
                                   const void* dt, const float* A_log, const void* B, const void* C, const float* D,
                                   const float* initial_states, const void* dy, const float* dfinal_states,
                                   void* dx, void* ddt, float* dA_log, void* dB, void* dC, float* dD,
                                   float* dinitial_states, void* workspace, size_t workspace_bytes, void* stream)
{
    size_t sub = 0, total = 0;
    int rc = varlen_plan(prob, seq_starts, &sub, &total);
    if (rc != SSD_OK) return rc;
    ssd::Shape s;
    {
        ssd_problem q = *prob;
        q.chunk_size = 256;
        if ((rc = ssd::validate(&q, true, &s)) != SSD_OK) return rc;
    }
    if (!x || !dt || !A_log || !B || !C || !dy || !dx || !ddt || !dA_log || !dB || !dC) return SSD_ERR_NULL_ARG;
    if (!aligned16(initial_states) || !aligned16(dfinal_states) || !aligned16(dinitial_states) ||
        !aligned16(x) || !aligned16(B) || !aligned16(C) || !aligned16(dy) || !aligned16(dx))
        return SSD_ERR_UNSUPPORTED_DIMS;   // (every slice below keeps the alignment: rows are multiples of 32 bytes)
    if (!workspace || workspace_bytes < total) return SSD_ERR_WORKSPACE;
    if (packed_backward_ok(prob)) {
        ssd::BwdParams p{};
        PackedBwdLayout pl{};
        if ((rc = packed_backward_plan(prob, &p, &pl)) != SSD_OK) return rc;
        char* ws = static_cast<char*>(workspace);
        p.x = x;
        p.dt = dt;
        p.A_log = A_log;
        p.B = B;
        p.C = C;
        p.D = D;
        p.init = initial_states;
        p.dy = dy;
        p.dfinal = dfinal_states;
        p.dx = dx;
        p.ddt = ddt;
        p.dA_log = dA_log;
        p.dB = dB;
        p.dC = dC;
        p.dD = D ? dD : nullptr;
        p.dinit = dinitial_states;
        p.hin = reinterpret_cast<float*>(ws + pl.l.hin);
        p.gnT = reinterpret_cast<float*>(ws + pl.l.gnT);
        p.dBp = reinterpret_cast<float*>(ws + pl.l.dBp);
        p.dCp = reinterpret_cast<float*>(ws + pl.l.dCp);
        p.dAp = reinterpret_cast<float*>(ws + pl.l.dAp);
        p.dDp = reinterpret_cast<float*>(ws + pl.l.dDp);
        int* starts = reinterpret_cast<int*>(ws + pl.starts);
        int4* vtab = reinterpret_cast<int4*>(ws + pl.vtab);
        int* seq_first = reinterpret_cast<int*>(ws + pl.seq_first);
        int* vcount = reinterpret_cast<int*>(ws + pl.vcount);
        p.vtab = vtab;
        p.seq_first = seq_first;
        p.vcount = vcount;
        ssd::SeqStartsArg arg;
        arg.n = static_cast<int>(prob->nseq);
        for (int64_t q = 0; q <= prob->nseq; ++q) arg.v[q] = static_cast<int>(seq_starts[q]);
        const hipStream_t st = static_cast<hipStream_t>(stream);
        hipError_t err = ssd::launch_seq_table(nullptr, &arg, p.T, p.nseq, static_cast<int>(ssd::kBwdQFast), p.nC, 1,
                                               starts, vtab, seq_first, vcount, st);
        if (err == hipSuccess) err = ssd::launch_backward_fast(p, st, nullptr, nullptr);
        return err == hipSuccess ? SSD_OK : SSD_ERR_LAUNCH;
    }
    const size_t act = s.bf16 ? 2 : 4;
    const int64_t H = s.H, HP = s.H * s.P, GN = s.G * s.N, HPN = s.H * s.P * s.N;
    float* partA = static_cast<float*>(workspace);
    float* partD = partA + prob->nseq * H;
    char* sub_ws = static_cast<char*>(workspace) + (total - sub);
    const auto at = [](const void* p, int64_t off) { return static_cast<const char*>(p) + off; };
    const auto atw = [](void* p, int64_t off) { return static_cast<char*>(p) + off; };
    for (int64_t q = 0; q < prob->nseq; ++q) {
        const int64_t t0 = seq_starts[q];
        ssd_problem pq = *prob;
        pq.seqlen = seq_starts[q + 1] - t0;
        rc = backward_impl(&pq, at(x, t0 * HP * act), at(dt, t0 * H * act), A_log, at(B, t0 * GN * act),
                           at(C, t0 * GN * act), D, initial_states ? initial_states + q * HPN : nullptr,
                           at(dy, t0 * HP * act), dfinal_states ? dfinal_states + q * HPN : nullptr,
                           atw(dx, t0 * HP * act), atw(ddt, t0 * H * act), partA + q * H, atw(dB, t0 * GN * act),
                           atw(dC, t0 * GN * act), D ? partD + q * H : nullptr,
                           dinitial_states ? dinitial_states + q * HPN : nullptr, sub_ws, sub, stream, nullptr,
                           nullptr);
        if (rc != SSD_OK) return SSD_ERR_LAUNCH;   // every check passed above: only a launch can fail here
    }
    const hipStream_t st = static_cast<hipStream_t>(stream);
    if (ssd::launch_sum_rows(partA, prob->nseq, H, dA_log, st) != hipSuccess) return SSD_ERR_LAUNCH;
    if (D && dD && ssd::launch_sum_rows(partD, prob->nseq, H, dD, st) != hipSuccess) return SSD_ERR_LAUNCH;
    return SSD_OK;
}

namespace {

// One launch over the whole packed row (the fused kernels' chunk table, the
// offsets handed over by value) where the shape and the number of sequences
// allow; else one call per sequence.  The varlen_per_sequence tuning forces
// the latter.
bool varlen_one_launch(const ssd_problem* prob)
{
    if (ssd::tuning(ssd::kTuneForceGeneral) == 1 || ssd::tuning(ssd::kTuneVarlenPerSequence) == 1) return false;
    ssd::Shape s;
    if (ssd::validate(prob, true, &s) != SSD_OK) return false;
    return ssd::fused_supported(s.P, s.N, s.Q, s.bf16) && fused_packed_ok(prob) && prob->nseq <= ssd::kArgSeqs;
}

int fwd_varlen_plan(const ssd_problem* prob, const int64_t* seq_starts, size_t* bytes)
{
    if (!prob || !seq_starts) return SSD_ERR_NULL_ARG;
    if (prob->batch != 1) return SSD_ERR_SEQIDX_BATCH;
    if (prob->nseq < 1 || prob->nseq > prob->seqlen) return SSD_ERR_BAD_SHAPE;
    if (seq_starts[0] != 0 || seq_starts[prob->nseq] != prob->seqlen) return SSD_ERR_BAD_SHAPE;
    for (int64_t s = 0; s < prob->nseq; ++s)
        if (seq_starts[s + 1] <= seq_starts[s]) return SSD_ERR_BAD_SHAPE;
    if (varlen_one_launch(prob)) {
        ssd::Shape sh;
        const int rc = ssd::validate(prob, true, &sh);
        if (rc != SSD_OK) return rc;
        *bytes = ssd::fused_layout(1, sh.T, sh.H, sh.N, sh.G, sh.nC, sh.nseq).total;
        return SSD_OK;
    }
    size_t need = 0;
    for (int64_t s = 0; s < prob->nseq; ++s) {
        ssd_problem q = *prob;
        q.seqlen = seq_starts[s + 1] - seq_starts[s];
        size_t b = 0;
        const int rc = ssd_workspace_bytes(&q, &b);
        if (rc != SSD_OK) return rc;
        if (b > need) need = b;
    }
    *bytes = need;
    return SSD_OK;
}

}  // namespace

extern "C" int ssd_forward_varlen_workspace_bytes(const ssd_problem* prob, const int64_t* seq_starts,
                                                  size_t* bytes)
{
    if (!bytes) return SSD_ERR_NULL_ARG;
    return fwd_varlen_plan(prob, seq_starts, bytes);
}

extern "C" int ssd_forward_varlen(const ssd_problem* prob, const int64_t* seq_starts, const void* x,
                                  const void* dt, const float* A_log, const void* B, const void* C,
                                  const float* D, const float* initial_states, void* y, float* final_states,
                                  void* workspace, size_t workspace_bytes, void* stream)
{
    size_t need = 0;
    int rc = fwd_varlen_plan(prob, seq_starts, &need);
    if (rc != SSD_OK) return rc;
    ssd::Shape s;
    if ((rc = ssd::validate(prob, true, &s)) != SSD_OK) return rc;
    if (!x || !dt || !A_log || !B || !C || !y) return SSD_ERR_NULL_ARG;
    if (!workspace || workspace_bytes < need) return SSD_ERR_WORKSPACE;
    if (varlen_one_launch(prob)) {
        ssd::SeqStartsArg a;
        a.n = static_cast<int>(prob->nseq);
        for (int64_t q = 0; q <= prob->nseq; ++q) a.v[q] = static_cast<int>(seq_starts[q]);
        return forward_impl(prob, nullptr, x, dt, A_log, B, C, D, initial_states, nullptr, y, final_states,
                            workspace, workspace_bytes, stream, nullptr, nullptr, &a);
    }
    const size_t act = s.bf16 ? 2 : 4;
    const int64_t H = s.H, HP = s.H * s.P, GN = s.G * s.N, HPN = s.H * s.P * s.N;
    for (int64_t q = 0; q < prob->nseq; ++q) {
        const int64_t t0 = seq_starts[q];
        ssd_problem pq = *prob;
        pq.seqlen = seq_starts[q + 1] - t0;
        rc = forward_impl(&pq, nullptr, static_cast<const char*>(x) + t0 * HP * act,
                          static_cast<const char*>(dt) + t0 * H * act, A_log,
                          static_cast<const char*>(B) + t0 * GN * act, static_cast<const char*>(C) + t0 * GN * act,
                          D, initial_states ? initial_states + q * HPN : nullptr, nullptr,
                          static_cast<char*>(y) + t0 * HP * act, final_states ? final_states + q * HPN : nullptr,
                          workspace, workspace_bytes, stream, nullptr, nullptr, nullptr, nullptr,
                          /*reset_status=*/q == 0);
        // the first call validates everything the later ones check (same shapes
        // but for seqlen): an error after it is a launch failure
        if (rc != SSD_OK) return q == 0 ? rc : SSD_ERR_LAUNCH;
    }
    return SSD_OK;
}

extern "C" const char* ssd_error_string(int code)
{
    switch (code) {
    case SSD_OK: return "success";
    case SSD_ERR_NULL_ARG: return "a required pointer is NULL";
    case SSD_ERR_BAD_SHAPE: return "invalid shape (dimension < 1, nheads % ngroups != 0, or bad nseq)";
    case SSD_ERR_BAD_CHUNK: return "chunk_size must be 32, 64, 128 or 256";
    case SSD_ERR_BAD_DTYPE: return "dtype must be SSD_DTYPE_F32 or SSD_DTYPE_BF16";
    case SSD_ERR_UNSUPPORTED_DIMS:
        return "headdim must be a multiple of 16 in [16,128] and dstate a multiple of 16 in [16,256]";
    case SSD_ERR_SEQIDX_BATCH: return "seq_idx requires batch == 1";
    case SSD_ERR_WORKSPACE: return "workspace missing or smaller than ssd_workspace_bytes()";
    case SSD_ERR_LAUNCH: return "kernel launch failed";
    case SSD_ERR_TOO_LARGE: return "problem exceeds the supported index range";
    case SSD_ERR_BAD_OPTION: return "option out of range (block option, or unknown tuning name or value)";
    case SSD_ERR_SCRATCH_TOO_SMALL:
        return "the problem needs more workspace than ssd_forward_noalloc's fixed scratch array";
    case SSD_ERR_STATE_TIMEOUT:
        return "a chunk's wait for the state of the chunk before it gave up: y and final_states are wrong";
    default: return "unknown ssd status";
    }
}

extern "C" int ssd_workspace_status(const void* workspace, void* stream)
{
    if (!workspace) return SSD_ERR_NULL_ARG;
    int word = 0;
    if (hipStreamSynchronize(static_cast<hipStream_t>(stream)) != hipSuccess ||
        hipMemcpy(&word, workspace, sizeof(int), hipMemcpyDeviceToHost) != hipSuccess)
        return SSD_ERR_LAUNCH;
    return word == 0 ? SSD_OK : SSD_ERR_STATE_TIMEOUT;
}

extern "C" int ssd_set_tuning(const char* name, int64_t value)
{
    if (!name) return SSD_ERR_NULL_ARG;
    struct Entry {
        const char* name;
        ssd::Tuning k;
        int64_t lo, hi;
    };
    static const Entry table[] = {
        {"force_general_path", ssd::kTuneForceGeneral, 0, 1},
        {"heads_per_item", ssd::kTuneHeadsPerItem, 0, 1 << 16},
        {"early_state_flag", ssd::kTuneEarlyFlag, 0, 2},
        {"max_workgroups", ssd::kTuneMaxWorkgroups, 0, 1 << 20},
        {"separate_block_post", ssd::kTuneSeparatePost, 0, 1},
        {"bwd_heads_per_slice", ssd::kTuneBwdHeadsPerSlice, 0, 1 << 16},
        {"varlen_per_sequence", ssd::kTuneVarlenPerSequence, 0, 1},
        {"state_wait_limit", ssd::kTuneStateWaitLimit, 0, INT64_MAX},
        {"fused_right_factor", ssd::kTuneFusedRightFactor, 0, 2},
        {"packed_order", ssd::kTunePackedOrder, 0, 2},
    };
    for (const Entry& e : table)
        if (std::strcmp(name, e.name) == 0) {
            if (value < e.lo || value > e.hi) return SSD_ERR_BAD_OPTION;
            ssd::g_tuning[e.k].store(value, std::memory_order_relaxed);
            return SSD_OK;
        }
    return SSD_ERR_BAD_OPTION;
}

// ---------------------------------------------------------------------------
// ssd_forward_noalloc: the forward with the library's own fixed workspace.
// The array lives in device memory of every GPU the library runs on; its name
// is only a host-side stand-in, so host code uses the address that
// hipGetSymbolAddress gives for the current device, never the name itself.
static __device__ __align__(256) unsigned char scratch[SSD_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices];   // per device, looked up once (under g_scratch_mu)

int scratch_address(void** out)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return SSD_ERR_LAUNCH;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return SSD_ERR_LAUNCH;
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return SSD_OK;
}

}  // namespace

extern "C" int ssd_forward_noalloc(const ssd_problem* prob, const void* x, const void* dt, const float* A_log,
                                   const void* B, const void* C, const float* D, const float* initial_states,
                                   const int32_t* seq_idx, void* y, float* final_states, int32_t* status,
                                   void* stream)
{
    size_t need = 0;
    int rc = ssd_workspace_bytes(prob, &need);   // host-side validation and sizing only
    if (rc != SSD_OK) return rc;
    if (need > SSD_NOALLOC_SCRATCH_BYTES) return SSD_ERR_SCRATCH_TOO_SMALL;
    void* ws = nullptr;
    if ((rc = scratch_address(&ws)) != SSD_OK) return rc;
    // the status word goes to the caller's pointer, or stays in the scratch header
    return forward_impl(prob, nullptr, x, dt, A_log, B, C, D, initial_states, seq_idx, y, final_states, ws,
                        SSD_NOALLOC_SCRATCH_BYTES, stream, nullptr, nullptr, nullptr, status);
}
