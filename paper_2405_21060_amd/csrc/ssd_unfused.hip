// Unfused SSD forward: one kernel per step of the block decomposition
// (Section 6), each contraction on the matrix cores.
//
//   k_chunk_prep    step 1: a = dt*A, chunk-local inclusive cumsum (log2 units),
//                           per-chunk scan coefficients (with sequence resets)
//   k_gram          C B^T per (batch, chunk, group), lower block triangle
//   k_chunk_state   right factors: chunk-final states from a zero start
//   k_varlen_final  packed rows: final states of sequences ending inside a chunk
//   k_state_scan    centre factors: scalar SSM scan over chunks, one thread per
//                   (batch, head, p, n) channel (Appendix B sequential mode)
//   k_chunk_output  diagonal block (L o C B^T) X plus left factors C h exp(cs)
//                   plus D x, stored in the activation dtype
//
// Conventions.  cs is in log2 units: cs2_t = log2(e) * sum_{k<=t} dt_k A within
// the chunk, so the 1-SS mask entry L_ts = exp(sum_{s<k<=t} a_k) is
// exp2(cs2_t - cs2_s).  A packed row splits a chunk into segments (maximal runs
// of one sequence id).  A segment "continues" when it starts at the chunk's
// first token and its sequence already ran in the previous chunk (or the chunk
// is the row's first); its incoming state is the state entering the chunk.
// Any other segment starts a sequence; its incoming state is that sequence's
// initial state, decayed from the segment start.
#include "ssd_device.h"
#include "ssd_internal.h"

namespace ssd {
namespace {

constexpr int kThreads = 256;  // 4 wavefronts
constexpr int kMaxQ = 256;
constexpr int kSlab = 32;      // tokens per staged K-step
constexpr int kPad = kSlab + 1;

// Sequence ids outside [0, nseq) break the seq_idx contract; state reads and
// writes for them are skipped so that such input cannot fault the device.
__device__ __forceinline__ bool unit_ok(const Params& p, int64_t u)
{
    return u >= 0 && u < p.nseq;
}

__device__ __forceinline__ int chunk_len(const Params& p, int c)
{
    const int64_t c0 = static_cast<int64_t>(c) * p.Q;
    return static_cast<int>(p.Q < p.T - c0 ? p.Q : p.T - c0);
}

// Per chunk and head: x4 = coefficient applied to the state at the chunk end,
// y = unit (sequence id, or batch row) of the chunk's last token,
// z = 1 when the last segment starts a sequence (reset), w = 1 when the
// chunk's last token is the last token of its unit.
// dt of token index `idx` of head h, after the block path's parameterisation
// (bias, softplus, clamp) when one is requested.
template <typename T>
__device__ __forceinline__ float load_dt(const Params& p, int64_t idx, int h)
{
    float v = Act<T>::load(static_cast<const T*>(p.dt), idx);
    if (p.dtx.active) {
        if (p.dtx.bias) v += p.dtx.bias[h];
        if (p.dtx.softplus) v = softplus_f(v);
        v = fminf(fmaxf(v, p.dtx.lo), p.dtx.hi);
    }
    return v;
}

template <typename T>
__global__ __launch_bounds__(kThreads) void k_chunk_prep(Params p)
{
    const int c = blockIdx.x, h = blockIdx.y, b = blockIdx.z, t = threadIdx.x;
    const int64_t c0 = static_cast<int64_t>(c) * p.Q;
    const int L = chunk_len(p, c);
    // this path has no bounded waits: its status is always fine
    if (p.status && c == 0 && h == 0 && b == 0 && t == 0) *p.status = 0;
    __shared__ float scr[kThreads / 64];
    __shared__ float cs_s[kThreads];
    __shared__ int q_s[kThreads];
    __shared__ int k0_s;

    const float A2 = -expf(p.A_log[h]) * kLog2e;
    float a2 = 0.f;
    if (t < L)
        a2 = load_dt<T>(p, (b * p.T + c0 + t) * p.H + h, h) * A2;
    const float cs = block_inclusive_scan(a2, scr);
    if (t < p.Q) p.cs[((b * p.H + h) * p.nC + c) * p.Q + t] = cs;
    cs_s[t] = cs;
    q_s[t] = (p.seq_idx && t < L) ? p.seq_idx[c0 + t] : 0;
    if (t == 0) k0_s = 0;
    __syncthreads();
    if (p.seq_idx && t > 0 && t < L && q_s[t] != q_s[t - 1]) atomicMax(&k0_s, t);
    __syncthreads();
    if (t == 0) {
        const int k0 = k0_s;
        int unit = b;
        int reset = 0;
        int ends = (c0 + L == p.T);
        if (p.seq_idx) {
            unit = q_s[L - 1];
            reset = (k0 > 0) || (c > 0 && p.seq_idx[c0 - 1] != q_s[0]);
            ends = ends || (p.seq_idx[c0 + L] != unit);
        }
        const float base = (reset && k0 > 0) ? cs_s[k0 - 1] : 0.f;
        const float coef = exp2f(cs_s[L - 1] - base);
        p.info[(b * p.H + h) * p.nC + c] = make_int4(__float_as_int(coef), unit, reset, ends);
    }
}

// G[t][s] = sum_n C_t[n] B_s[n] for 16x16 tiles with s-tile <= t-tile.
template <typename T>
__global__ __launch_bounds__(kThreads) void k_gram(Params p)
{
    const int c = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, r = lane & 15, lg = lane >> 4;
    const int64_t c0 = static_cast<int64_t>(c) * p.Q;
    const int L = chunk_len(p, c);
    const int nq = static_cast<int>(p.Q / 16);
    const int ntile = nq * (nq + 1) / 2;
    const T* Bp = static_cast<const T*>(p.B);
    const T* Cp = static_cast<const T*>(p.C);
    float* Gp = p.gram + ((b * p.G + g) * p.nC + c) * p.Q * p.Q;
    for (int tau = wave; tau < ntile; tau += kThreads / 64) {
        int i = 0;
        while ((i + 1) * (i + 2) / 2 <= tau) ++i;
        const int j = tau - i * (i + 1) / 2;
        const int t = 16 * i + r, s = 16 * j + r;
        f32x4_t acc = zero4();
        for (int k0 = 0; k0 < p.N; k0 += 32) {
            Frag8 fa, fb;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int n = k0 + 8 * lg + e;
                fa.v[e] = (t < L && n < p.N) ? Act<T>::load(Cp, ((b * p.T + c0 + t) * p.G + g) * p.N + n) : 0.f;
                fb.v[e] = (s < L && n < p.N) ? Act<T>::load(Bp, ((b * p.T + c0 + s) * p.G + g) * p.N + n) : 0.f;
            }
            acc = mma_step(fa, fb, acc, T());
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) Gp[(16 * i + 4 * lg + v) * p.Q + 16 * j + r] = acc[v];
    }
}

// Sum over the tokens s of [st, en] of w_s x_s B_s^T into a (P x N) tile set,
// w_s = dt_s exp2(cs2_en - cs2_s); the result (plus hin_scale * hin, when hin
// is given) is stored to dst (P x N, row-major).  Block-uniform call.
template <typename T>
__device__ void segment_state(const Params& p, int b, int c, int h, int g, int st, int en,
                              const float* cs_s, const float* dt_s, float* w_s, float* xT,
                              float* BT, float* dst, const float* hin, float hin_scale)
{
    constexpr int kMaxTiles = 32;  // (128/16) * (256/16) / 4 waves
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, r = lane & 15, lg = lane >> 4;
    const int P = static_cast<int>(p.P), N = static_cast<int>(p.N);
    const int TN = N / 16, ntiles = (P / 16) * TN;
    const int64_t c0 = static_cast<int64_t>(c) * p.Q;
    const T* xp = static_cast<const T*>(p.x);
    const T* Bp = static_cast<const T*>(p.B);

    for (int t = threadIdx.x; t < kMaxQ; t += kThreads)
        w_s[t] = (t >= st && t <= en) ? dt_s[t] * exp2f(cs_s[en] - cs_s[t]) : 0.f;
    __syncthreads();

    f32x4_t acc[kMaxTiles];
#pragma unroll
    for (int k = 0; k < kMaxTiles; ++k) acc[k] = zero4();

    for (int s0 = (st / kSlab) * kSlab; s0 <= en; s0 += kSlab) {
        for (int idx = threadIdx.x; idx < kSlab * P; idx += kThreads) {
            const int ss = idx / P, pp = idx % P, s = s0 + ss;
            xT[pp * kPad + ss] = (s <= en) ? Act<T>::load(xp, ((b * p.T + c0 + s) * p.H + h) * p.P + pp) * w_s[s] : 0.f;
        }
        for (int idx = threadIdx.x; idx < kSlab * N; idx += kThreads) {
            const int ss = idx / N, n = idx % N, s = s0 + ss;
            BT[n * kPad + ss] = (s <= en) ? Act<T>::load(Bp, ((b * p.T + c0 + s) * p.G + g) * p.N + n) : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < kMaxTiles; ++k) {
            const int tau = wave + 4 * k;
            if (tau < ntiles) {
                const int pt = tau / TN, nt = tau % TN;
                Frag8 fa, fb;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    fa.v[e] = xT[(16 * pt + r) * kPad + 8 * lg + e];
                    fb.v[e] = BT[(16 * nt + r) * kPad + 8 * lg + e];
                }
                acc[k] = mma_step(fa, fb, acc[k], T());
            }
        }
        __syncthreads();
    }
#pragma unroll
    for (int k = 0; k < kMaxTiles; ++k) {
        const int tau = wave + 4 * k;
        if (tau < ntiles) {
            const int pt = tau / TN, nt = tau % TN;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int pp = 16 * pt + 4 * lg + v, n = 16 * nt + r;
                float val = acc[k][v];
                if (hin) val += hin_scale * hin[pp * N + n];
                dst[pp * N + n] = val;
            }
        }
    }
    __syncthreads();
}

// Shared-memory staging of one chunk's per-token scalars.
struct ChunkScalars {
    float cs[kMaxQ], dt[kMaxQ], w[kMaxQ];
    int q[kMaxQ];
};

template <typename T>
__device__ __forceinline__ void load_chunk_scalars(const Params& p, int b, int c, int h, int L,
                                                   ChunkScalars& sh)
{
    const int t = threadIdx.x;
    const int64_t c0 = static_cast<int64_t>(c) * p.Q;
    if (t < L) {
        sh.cs[t] = p.cs[((b * p.H + h) * p.nC + c) * p.Q + t];
        sh.dt[t] = load_dt<T>(p, (b * p.T + c0 + t) * p.H + h, h);
        sh.q[t] = p.seq_idx ? p.seq_idx[c0 + t] : 0;
    }
    __syncthreads();
}

// Right factors: the chunk's state at its last token from a zero start,
// restricted to the chunk's last segment.
template <typename T>
__global__ __launch_bounds__(kThreads) void k_chunk_state(Params p)
{
    const int c = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
    const int g = static_cast<int>(h / (p.H / p.G));
    const int L = chunk_len(p, c);
    __shared__ ChunkScalars sh;
    __shared__ float xT[128 * kPad];
    __shared__ float BT[256 * kPad];
    load_chunk_scalars<T>(p, b, c, h, L, sh);
    int st = 0;
    if (p.seq_idx)
        for (int k = L - 1; k > 0; --k)
            if (sh.q[k - 1] != sh.q[k]) { st = k; break; }
    float* dst = p.states + ((b * p.nC + c) * p.H + h) * p.P * p.N;
    segment_state<T>(p, b, c, h, g, st, L - 1, sh.cs, sh.dt, sh.w, xT, BT, dst, nullptr, 0.f);
}

// Packed rows: final states of sequences that end before their chunk's last
// token (those ending on a chunk's last token come out of the scan).
template <typename T>
__global__ __launch_bounds__(kThreads) void k_varlen_final(Params p)
{
    const int c = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
    const int g = static_cast<int>(h / (p.H / p.G));
    const int64_t c0 = static_cast<int64_t>(c) * p.Q;
    const int L = chunk_len(p, c);
    const int64_t PN = p.P * p.N;
    __shared__ ChunkScalars sh;
    __shared__ float xT[128 * kPad];
    __shared__ float BT[256 * kPad];
    load_chunk_scalars<T>(p, b, c, h, L, sh);
    int st = 0;
    for (int en = 0; en < L - 1; ++en) {
        if (sh.q[en] == sh.q[en + 1]) continue;
        const int q = sh.q[en];
        const bool cont = (st == 0) && (c == 0 || p.seq_idx[c0 - 1] == q);
        const float* hin = cont ? p.states + ((b * p.nC + c) * p.H + h) * PN
                                : (p.init && unit_ok(p, q) ? p.init + (static_cast<int64_t>(q) * p.H + h) * PN : nullptr);
        const float base = (st > 0) ? sh.cs[st - 1] : 0.f;
        if (!unit_ok(p, q)) { st = en + 1; continue; }
        segment_state<T>(p, b, c, h, g, st, en, sh.cs, sh.dt, sh.w, xT, BT,
                         p.fin + (static_cast<int64_t>(q) * p.H + h) * PN, hin,
                         exp2f(sh.cs[en] - base));
        st = en + 1;
    }
}

// h_{-1} = initial state of the row (or of the first sequence); per chunk:
// store the entering state over the chunk state, then h = coef h + S (or
// coef * init[unit] + S after a reset); write final states at unit ends.
__global__ __launch_bounds__(kThreads) void k_state_scan(Params p)
{
    const int64_t PN = p.P * p.N;
    const int64_t idx = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    const int h = blockIdx.y, b = blockIdx.z;
    if (idx >= PN) return;
    float hs = 0.f;
    if (p.init) {
        const int64_t u0 = p.seq_idx ? p.seq_idx[0] : b;
        if (unit_ok(p, u0)) hs = p.init[(u0 * p.H + h) * PN + idx];
    }
    for (int64_t c = 0; c < p.nC; ++c) {
        const int4 inf = p.info[(b * p.H + h) * p.nC + c];
        float* slot = p.states + ((b * p.nC + c) * p.H + h) * PN + idx;
        const float S = *slot;
        *slot = hs;
        const float coef = __int_as_float(inf.x);
        const bool uok = unit_ok(p, inf.y);
        if (inf.z)
            hs = (p.init && uok ? coef * p.init[(static_cast<int64_t>(inf.y) * p.H + h) * PN + idx] : 0.f) + S;
        else
            hs = coef * hs + S;
        if (inf.w && p.fin && uok) p.fin[(static_cast<int64_t>(inf.y) * p.H + h) * PN + idx] = hs;
    }
}

template <typename T>
__global__ __launch_bounds__(kThreads) void k_chunk_output(Params p)
{
    constexpr int kMaxStrips = kMaxQ / 16 / 4;  // strips of 16 rows per wave
    constexpr int kMaxPT = 128 / 16;
    const int c = blockIdx.x, h = blockIdx.y, b = blockIdx.z, t0 = threadIdx.x;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, r = lane & 15, lg = lane >> 4;
    const int g = static_cast<int>(h / (p.H / p.G));
    const int64_t c0 = static_cast<int64_t>(c) * p.Q;
    const int L = chunk_len(p, c);
    const int P = static_cast<int>(p.P), N = static_cast<int>(p.N);
    const int TP = P / 16, nq = static_cast<int>(p.Q / 16);
    const int64_t PN = p.P * p.N;
    const T* xp = static_cast<const T*>(p.x);
    const T* Cp = static_cast<const T*>(p.C);
    const float* Gp = p.gram + ((b * p.G + g) * p.nC + c) * p.Q * p.Q;
    __shared__ float cs_s[kMaxQ], dt_s[kMaxQ];
    __shared__ int q_s[kMaxQ];
    __shared__ float xT[128 * kPad];

    if (t0 < kMaxQ) {
        const bool in = t0 < L;
        cs_s[t0] = in ? p.cs[((b * p.H + h) * p.nC + c) * p.Q + t0] : 0.f;
        dt_s[t0] = in ? load_dt<T>(p, (b * p.T + c0 + t0) * p.H + h, h) : 0.f;
        q_s[t0] = (p.seq_idx && in) ? p.seq_idx[c0 + t0] : 0;
    }
    __syncthreads();

    f32x4_t acc[kMaxStrips][kMaxPT];
#pragma unroll
    for (int si = 0; si < kMaxStrips; ++si)
#pragma unroll
        for (int pt = 0; pt < kMaxPT; ++pt) acc[si][pt] = zero4();

    // diagonal block: Y^T[p][t] = sum_s x^T[p][s] * (G[t][s] L_ts dt_s)
    for (int s0 = 0; s0 < L; s0 += kSlab) {
        for (int idx = threadIdx.x; idx < kSlab * P; idx += kThreads) {
            const int ss = idx / P, pp = idx % P, s = s0 + ss;
            xT[pp * kPad + ss] = (s < L) ? Act<T>::load(xp, ((b * p.T + c0 + s) * p.H + h) * p.P + pp) : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int si = 0; si < kMaxStrips; ++si) {
            const int i = wave + 4 * si;
            if (i < nq && 16 * i + 15 >= s0) {
                const int t = 16 * i + r;
                Frag8 fb;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int s = s0 + 8 * lg + e;
                    const bool on = (s <= t) && (t < L) && (q_s[s] == q_s[t]);
                    fb.v[e] = on ? Gp[t * p.Q + s] * exp2f(cs_s[t] - cs_s[s]) * dt_s[s] : 0.f;
                }
#pragma unroll
                for (int pt = 0; pt < kMaxPT; ++pt) {
                    if (pt < TP) {
                        Frag8 fa;
#pragma unroll
                        for (int e = 0; e < 8; ++e) fa.v[e] = xT[(16 * pt + r) * kPad + 8 * lg + e];
                        acc[si][pt] = mma_step(fa, fb, acc[si][pt], T());
                    }
                }
            }
        }
        __syncthreads();
    }

    // left factors: per segment, Y^T[p][t] += scale_t * sum_n hin[p][n] C_t[n]
    int st = 0;
    while (st < L) {
        int en = st;
        while (en + 1 < L && q_s[en + 1] == q_s[st]) ++en;
        const int q = q_s[st];
        const bool cont = (st == 0) && (c == 0 || !p.seq_idx || p.seq_idx[c0 - 1] == q);
        const float* hin = cont ? p.states + ((b * p.nC + c) * p.H + h) * PN
                                : (p.init && unit_ok(p, q) ? p.init + (static_cast<int64_t>(q) * p.H + h) * PN : nullptr);
        const float base = (st > 0) ? cs_s[st - 1] : 0.f;
        if (hin) {
#pragma unroll
            for (int si = 0; si < kMaxStrips; ++si) {
                const int i = wave + 4 * si;
                if (i < nq && 16 * i + 15 >= st && 16 * i <= en) {
                    const int t = 16 * i + r;
                    const float scale = (t >= st && t <= en) ? exp2f(cs_s[t] - base) : 0.f;
#pragma unroll
                    for (int pt = 0; pt < kMaxPT; ++pt) {
                        if (pt < TP) {
                            f32x4_t tmp = zero4();
                            for (int k0 = 0; k0 < N; k0 += 32) {
                                Frag8 fa, fb;
#pragma unroll
                                for (int e = 0; e < 8; ++e) {
                                    const int n = k0 + 8 * lg + e;
                                    fa.v[e] = (n < N) ? hin[(16 * pt + r) * N + n] : 0.f;
                                    fb.v[e] = (n < N && t < L) ? Act<T>::load(Cp, ((b * p.T + c0 + t) * p.G + g) * p.N + n) : 0.f;
                                }
                                tmp = mma_step(fa, fb, tmp, T());
                            }
#pragma unroll
                            for (int v = 0; v < 4; ++v) acc[si][pt][v] += scale * tmp[v];
                        }
                    }
                }
            }
        }
        st = en + 1;
    }

    // skip term and store
    const float Dh = p.D ? p.D[h] : 0.f;
    T* yp = static_cast<T*>(p.y);
#pragma unroll
    for (int si = 0; si < kMaxStrips; ++si) {
        const int i = wave + 4 * si;
        const int t = 16 * i + r;
        if (i < nq && t < L) {
#pragma unroll
            for (int pt = 0; pt < kMaxPT; ++pt) {
                if (pt < TP) {
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const int pp = 16 * pt + 4 * lg + v;
                        const int64_t o = ((b * p.T + c0 + t) * p.H + h) * p.P + pp;
                        Act<T>::store(yp, o, acc[si][pt][v] + Dh * Act<T>::load(xp, o));
                    }
                }
            }
        }
    }
}

template <typename T>
hipError_t launch_all(const Params& p, hipStream_t stream, hipEvent_t ev_begin, hipEvent_t ev_end)
{
    const dim3 blk(kThreads);
    const dim3 g_chunk(static_cast<unsigned>(p.nC), static_cast<unsigned>(p.H), static_cast<unsigned>(p.b));
    const dim3 g_gram(static_cast<unsigned>(p.nC), static_cast<unsigned>(p.G), static_cast<unsigned>(p.b));
    const dim3 g_scan(static_cast<unsigned>((p.P * p.N + kThreads - 1) / kThreads),
                      static_cast<unsigned>(p.H), static_cast<unsigned>(p.b));
    hipLaunchKernelGGL(k_chunk_prep<T>, g_chunk, blk, 0, stream, p);
    hipLaunchKernelGGL(k_gram<T>, g_gram, blk, 0, stream, p);
    hipLaunchKernelGGL(k_chunk_state<T>, g_chunk, blk, 0, stream, p);
    hipLaunchKernelGGL(k_state_scan, g_scan, blk, 0, stream, p);
    hipError_t err = hipGetLastError();
    if (err == hipSuccess && ev_begin) err = hipEventRecord(ev_begin, stream);
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(k_chunk_output<T>, g_chunk, blk, 0, stream, p);
    err = hipGetLastError();
    if (err == hipSuccess && ev_end) err = hipEventRecord(ev_end, stream);
    if (err != hipSuccess) return err;
    if (p.seq_idx && p.fin) hipLaunchKernelGGL(k_varlen_final<T>, g_chunk, blk, 0, stream, p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_unfused(const Params& p, bool bf16, hipStream_t stream, hipEvent_t ev_begin,
                          hipEvent_t ev_end)
{
    return bf16 ? launch_all<uint16_t>(p, stream, ev_begin, ev_end)
                : launch_all<float>(p, stream, ev_begin, ev_end);
}

}  // namespace ssd
