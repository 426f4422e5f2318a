// Gradients of the SSD layer, in the chunked form of the adjoint of its
// recurrence.  The paper gives the layer's training cost (Section 6.3) but no
// backward algorithm; this is the reverse-mode derivative of the chunked block
// decomposition of Section 6, chunk by chunk.
//
// Per (batch row, head), with chunks of Q = kBwdQ tokens, a_t = dt_t A,
// cs_t = chunk-local inclusive sum of a, e(u,t) = exp(cs_u - cs_t) (u >= t),
// X~_t = dt_t x_t, h_in the state entering the chunk, h_out the state leaving
// it and Gn the gradient of the loss with respect to h_out:
//
//   states      H_c = sum_s e(end,s) X~_s B_s^T           (h_out = exp(cs_end) h_in + H_c)
//               W_c = sum_u exp(cs_u) dy_u C_u^T          (what the chunk's outputs add to
//                                                          the gradient of h_in)
//   scans       h_in(c+1) = exp(cs_end(c)) h_in(c) + H_c,     from the initial state
//               Gn(c-1)   = exp(cs_end(c)) Gn(c) + W_c,       from the final-state gradient;
//               the gradient of the initial state is exp(cs_end(0)) Gn(0) + W_0
//   chunk       with G0(u,t) = C_u . B_t, R0(u,t) = dy_u . X~_t,
//               Gs = e G0, Rs = e R0, l(u,t) = e G0 R0 (all for u >= t):
//     dX~_t = sum_u Gs(u,t) dy_u + e(end,t) Gn B_t,       dx_t = dt_t dX~_t + D dy_t
//     dB_t  = sum_u Rs(u,t) C_u  + e(end,t) Gn^T X~_t     (summed over a group's heads)
//     dC_u  = sum_t Rs(u,t) B_t  + exp(cs_u) h_in^T dy_u  (summed over a group's heads)
//     dcs_t = sum_s l(t,s) - sum_u l(u,t) + exp(cs_t) dy_t . (h_in C_t)
//             - e(end,t) X~_t . (Gn B_t) + [t = end] <Gn, h_out>,
//     <Gn, h_out> = exp(cs_end) <Gn, h_in> + sum_s e(end,s) X~_s . (Gn B_s),
//     da_k = sum_{t >= k} dcs_t,  ddt_k = x_k . dX~_k + A da_k,
//     dA = sum dt_k da_k,  dA_log = A dA,  dD = sum dy . x.
//
// Kernels: k_bwd_states (cumsum, H_c, W_c), k_bwd_scan (both scans),
// k_bwd_chunk (everything per chunk; a workgroup walks a slice of a group's
// heads, which share B, C and G0, and accumulates dB and dC over them),
// k_bwd_reduce_bc and k_bwd_reduce_head (sums over slices, chunks and rows in
// a fixed order: results are deterministic).  Float32 FMAs throughout.
#include "ssd_bwd.h"
#include "ssd_device.h"

namespace ssd {
namespace {

constexpr int kQ = static_cast<int>(kBwdQ);
constexpr int kThreads = 256;
constexpr int kTpt = kThreads / kQ;      // threads per token in the chunk kernel (8)

template <typename T>
__device__ __forceinline__ float ld(const void* p, int64_t i) { return Act<T>::load(static_cast<const T*>(p), i); }

template <typename T>
__device__ __forceinline__ void st(void* p, int64_t i, float v) { Act<T>::store(static_cast<T*>(p), i, v); }

__device__ __forceinline__ int chunk_len(int64_t T, int64_t c)
{
    const int64_t r = T - c * kQ;
    return static_cast<int>(r < kQ ? r : kQ);
}

// Sum over the 256 threads of the block in a fixed order.
__device__ __forceinline__ float block_sum256(float v, float* scr)
{
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    if ((threadIdx.x & 63) == 0) scr[threadIdx.x >> 6] = v;
    __syncthreads();
    const float s = (scr[0] + scr[1]) + (scr[2] + scr[3]);
    __syncthreads();
    return s;
}

// Per (chunk, batch row, head): the chunk's cumsum and its two state-sized
// terms H_c (into hin) and W_c (into gn).  Shared memory: the weighted
// operands, Q x P twice and Q x N twice.
template <typename T>
__global__ __launch_bounds__(kThreads) void k_bwd_states(BwdParams p)
{
    extern __shared__ __attribute__((aligned(16))) float sm[];
    const int P = static_cast<int>(p.P), N = static_cast<int>(p.N);
    float* sXw = sm;               // e(end,s) dt_s x_s
    float* sDw = sXw + kQ * P;     // exp(cs_u) dy_u
    float* sB = sDw + kQ * P;
    float* sC = sB + kQ * N;
    __shared__ float scs[kQ], sdt[kQ];

    const int64_t c = blockIdx.x, b = blockIdx.y, h = blockIdx.z;
    const int64_t g = h / (p.H / p.G);
    const int L = chunk_len(p.T, c);
    const int tid = threadIdx.x;
    const int64_t t0 = b * p.T + c * kQ;   // flat token index of the chunk's first token
    const int64_t bh = b * p.H + h;

    if (tid < 64) {
        // inclusive cumsum of dt*A (log2 units) over the chunk, one wavefront
        const float A2 = -expf(p.A_log[h]) * kLog2e;
        const float dtv = tid < L ? ld<T>(p.dt, (t0 + tid) * p.H + h) : 0.f;
        float v = dtv * A2;
        for (int sh = 1; sh < 64; sh <<= 1) {
            const float o = __shfl_up(v, sh, 64);
            if (tid >= sh) v += o;
        }
        if (tid < kQ) {
            scs[tid] = v;
            sdt[tid] = dtv;
            p.cs[(bh * p.nC + c) * kQ + tid] = v;
        }
    }
    __syncthreads();
    const float csend = scs[L - 1];
    for (int i = tid; i < kQ * P; i += kThreads) {
        const int s = i / P, pr = i - s * P;
        float xw = 0.f, dw = 0.f;
        if (s < L) {
            const int64_t xi = ((t0 + s) * p.H + h) * p.P + pr;
            xw = exp2f(csend - scs[s]) * sdt[s] * ld<T>(p.x, xi);
            dw = exp2f(scs[s]) * ld<T>(p.dy, xi);
        }
        sXw[i] = xw;
        sDw[i] = dw;
    }
    for (int i = tid; i < kQ * N; i += kThreads) {
        const int s = i / N, n = i - s * N;
        float bv = 0.f, cv = 0.f;
        if (s < L) {
            const int64_t bi = ((t0 + s) * p.G + g) * p.N + n;
            bv = ld<T>(p.B, bi);
            cv = ld<T>(p.C, bi);
        }
        sB[i] = bv;
        sC[i] = cv;
    }
    __syncthreads();
    const int64_t base = ((b * p.nC + c) * p.H + h) * p.P * p.N;
    for (int i = tid; i < P * N; i += kThreads) {
        const int pr = i / N, n = i - pr * N;
        float hs = 0.f, ws = 0.f;
        for (int s = 0; s < L; ++s) {
            hs = fmaf(sXw[s * P + pr], sB[s * N + n], hs);
            ws = fmaf(sDw[s * P + pr], sC[s * N + n], ws);
        }
        p.hin[base + i] = hs;
        p.gn[base + i] = ws;
    }
}

// Both scans over chunks, one thread per 4 consecutive state elements of one
// (batch row, head).  In place: hin(c) <- state entering chunk c,
// gn(c) <- gradient of the state leaving chunk c; writes dinit.
__global__ __launch_bounds__(kThreads) void k_bwd_scan(BwdParams p)
{
    const int64_t PN4 = p.P * p.N / 4;
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (i >= p.b * p.H * PN4) return;
    const int64_t bh = i / PN4, e4 = i - bh * PN4;
    const int64_t b = bh / p.H, h = bh - b * p.H;
    const int64_t stride = p.H * PN4;       // between consecutive chunks, in float4
    float4* hin = reinterpret_cast<float4*>(p.hin) + (b * p.nC * p.H + h) * PN4 + e4;
    float4* gn = reinterpret_cast<float4*>(p.gn) + (b * p.nC * p.H + h) * PN4 + e4;
    const float* cs = p.cs + bh * p.nC * kQ;

    float4 acc = p.init ? reinterpret_cast<const float4*>(p.init)[i] : make_float4(0.f, 0.f, 0.f, 0.f);
    for (int64_t c = 0; c < p.nC; ++c) {
        const float a = exp2f(cs[c * kQ + chunk_len(p.T, c) - 1]);
        const float4 loc = hin[c * stride];
        hin[c * stride] = acc;
        acc.x = fmaf(a, acc.x, loc.x);
        acc.y = fmaf(a, acc.y, loc.y);
        acc.z = fmaf(a, acc.z, loc.z);
        acc.w = fmaf(a, acc.w, loc.w);
    }
    acc = p.dfinal ? reinterpret_cast<const float4*>(p.dfinal)[i] : make_float4(0.f, 0.f, 0.f, 0.f);
    for (int64_t c = p.nC - 1; c >= 0; --c) {
        const float a = exp2f(cs[c * kQ + chunk_len(p.T, c) - 1]);
        const float4 loc = gn[c * stride];
        gn[c * stride] = acc;
        acc.x = fmaf(a, acc.x, loc.x);
        acc.y = fmaf(a, acc.y, loc.y);
        acc.z = fmaf(a, acc.z, loc.z);
        acc.w = fmaf(a, acc.w, loc.w);
    }
    if (p.dinit) reinterpret_cast<float4*>(p.dinit)[i] = acc;
}

constexpr int kMaxNk = 256 / kTpt;   // n values per thread at the largest dstate (32)

// Per (chunk, batch row, group, head slice): the chunk terms of every
// gradient (formulas at the top of the file).  Thread layout: token
// t = tid / 8, lane j = tid % 8 of the token's eight; feature index
// f = j + 8 k for the k-th value a thread holds.
template <typename T>
__global__ __launch_bounds__(kThreads) void k_bwd_chunk(BwdParams p)
{
    extern __shared__ __attribute__((aligned(16))) float sm[];
    const int P = static_cast<int>(p.P), N = static_cast<int>(p.N);
    float* sB = sm;                  // Q x N
    float* sC = sB + kQ * N;         // Q x N
    float* sx = sC + kQ * N;         // Q x P   x (raw)
    float* sdy = sx + kQ * P;        // Q x P
    float* sG0 = sdy + kQ * P;       // Q x Q   C_u . B_t (u >= t)
    float* sGs = sG0 + kQ * kQ;      // Q x Q
    float* sRs = sGs + kQ * kQ;      // Q x Q
    float* sL = sRs + kQ * kQ;       // Q x Q
    __shared__ float scs[kQ], sdt[kQ], seend[kQ], sxdx[kQ], sq1[kQ], sq2[kQ], sdyx[kQ], sdcs[kQ];
    __shared__ float scr[4];

    const int64_t c = blockIdx.x, b = blockIdx.y;
    const int64_t g = blockIdx.z / p.S, slice = blockIdx.z - g * p.S;
    const int64_t hpg = p.H / p.G;
    const int64_t h_lo = g * hpg + slice * p.hs;
    const int64_t h_hi = (slice + 1) * p.hs < hpg ? h_lo + p.hs : g * hpg + hpg;
    const int L = chunk_len(p.T, c);
    const int tid = threadIdx.x;
    const int tt = tid / kTpt, j = tid - tt * kTpt;
    const int64_t t0 = b * p.T + c * kQ;
    const int nk = N / kTpt, pk = P / kTpt;

    for (int i = tid; i < kQ * N; i += kThreads) {
        const int s = i / N, n = i - s * N;
        float bv = 0.f, cv = 0.f;
        if (s < L) {
            const int64_t bi = ((t0 + s) * p.G + g) * p.N + n;
            bv = ld<T>(p.B, bi);
            cv = ld<T>(p.C, bi);
        }
        sB[i] = bv;
        sC[i] = cv;
    }
    __syncthreads();
    for (int k = 0; k < kQ / kTpt; ++k) {
        const int u = tt, t = j + kTpt * k;
        float acc = 0.f;
        if (t <= u && u < L)
            for (int n = 0; n < N; ++n) acc = fmaf(sC[u * N + n], sB[t * N + n], acc);
        sG0[u * kQ + t] = acc;
    }

    float dBacc[kMaxNk], dCacc[kMaxNk];
#pragma unroll
    for (int k = 0; k < kMaxNk; ++k) dBacc[k] = dCacc[k] = 0.f;

    for (int64_t h = h_lo; h < h_hi; ++h) {
        const int64_t bh = b * p.H + h;
        const float Ah = -expf(p.A_log[h]);
        const float Dh = p.D ? p.D[h] : 0.f;
        const float* Gn = p.gn + ((b * p.nC + c) * p.H + h) * p.P * p.N;
        const float* Hin = p.hin + ((b * p.nC + c) * p.H + h) * p.P * p.N;
        __syncthreads();   // previous head done with the per-head shared arrays
        for (int i = tid; i < kQ * P; i += kThreads) {
            const int s = i / P, pr = i - s * P;
            float xv = 0.f, dv = 0.f;
            if (s < L) {
                const int64_t xi = ((t0 + s) * p.H + h) * p.P + pr;
                xv = ld<T>(p.x, xi);
                dv = ld<T>(p.dy, xi);
            }
            sx[i] = xv;
            sdy[i] = dv;
        }
        if (tid < kQ) {
            const float csv = p.cs[(bh * p.nC + c) * kQ + tid];
            scs[tid] = csv;
            sdt[tid] = tid < L ? ld<T>(p.dt, (t0 + tid) * p.H + h) : 0.f;
        }
        __syncthreads();
        const float csend = scs[L - 1];
        if (tid < kQ) seend[tid] = tid < L ? exp2f(csend - scs[tid]) : 0.f;

        // scores for the pairs u = tt, t = j + 8 k
        for (int k = 0; k < kQ / kTpt; ++k) {
            const int u = tt, t = j + kTpt * k;
            float gs = 0.f, rs = 0.f, l = 0.f;
            if (t <= u && u < L) {
                float r0 = 0.f;
                for (int pr = 0; pr < P; ++pr) r0 = fmaf(sdy[u * P + pr], sx[t * P + pr], r0);
                r0 *= sdt[t];
                const float e = exp2f(scs[u] - scs[t]);
                gs = e * sG0[u * kQ + t];
                rs = e * r0;
                l = gs * r0;
            }
            sGs[u * kQ + t] = gs;
            sRs[u * kQ + t] = rs;
            sL[u * kQ + t] = l;
        }
        // <Gn, h_in>
        float gh = 0.f;
        for (int i = tid; i < P * N; i += kThreads) gh = fmaf(Gn[i], Hin[i], gh);
        gh = block_sum256(gh, scr);   // also orders the score stores before their use

        // dX~ and dx for (t = tt, p = j + 8 k); per-token sums over p
        {
            const int t = tt;
            float sxd = 0.f, sxgb = 0.f, sdyhc = 0.f, sdyx_ = 0.f;
            if (t < L) {
                const float dtv = sdt[t], ee = seend[t];
                for (int k = 0; k < pk; ++k) {
                    const int pr = j + kTpt * k;
                    float dX = 0.f;
                    for (int u = t; u < L; ++u) dX = fmaf(sGs[u * kQ + t], sdy[u * P + pr], dX);
                    float gb = 0.f, hc = 0.f;
                    const float* gr = Gn + static_cast<int64_t>(pr) * N;
                    const float* hr = Hin + static_cast<int64_t>(pr) * N;
                    for (int n = 0; n < N; ++n) {
                        gb = fmaf(gr[n], sB[t * N + n], gb);
                        hc = fmaf(hr[n], sC[t * N + n], hc);
                    }
                    dX = fmaf(ee, gb, dX);
                    const float xv = sx[t * P + pr], dyv = sdy[t * P + pr];
                    sxd = fmaf(xv, dX, sxd);
                    sxgb = fmaf(xv, gb, sxgb);
                    sdyhc = fmaf(dyv, hc, sdyhc);
                    sdyx_ = fmaf(dyv, xv, sdyx_);
                    st<T>(p.dx, ((t0 + t) * p.H + h) * p.P + pr, fmaf(dtv, dX, Dh * dyv));
                }
            }
            for (int off = 1; off < kTpt; off <<= 1) {
                sxd += __shfl_xor(sxd, off, 64);
                sxgb += __shfl_xor(sxgb, off, 64);
                sdyhc += __shfl_xor(sdyhc, off, 64);
                sdyx_ += __shfl_xor(sdyx_, off, 64);
            }
            if (j == 0) {
                sxdx[t] = sxd;
                sq2[t] = t < L ? sdt[t] * sxgb : 0.f;   // X~_t . (Gn B_t)
                sq1[t] = sdyhc;                           // dy_t . (h_in C_t)
                sdyx[t] = sdyx_;
            }
        }

        // dB and dC for (t = tt, n = j + 8 k)
        {
            const int t = tt;
            if (t < L) {
                const float ee = seend[t] * sdt[t], ec = exp2f(scs[t]);
#pragma unroll
                for (int k = 0; k < kMaxNk; ++k) {
                    if (k >= nk) break;
                    const int n = j + kTpt * k;
                    float db = 0.f, dc = 0.f;
                    for (int u = t; u < L; ++u) db = fmaf(sRs[u * kQ + t], sC[u * N + n], db);
                    for (int s = 0; s <= t; ++s) dc = fmaf(sRs[t * kQ + s], sB[s * N + n], dc);
                    float xg = 0.f, dh = 0.f;
                    for (int pr = 0; pr < P; ++pr) {
                        xg = fmaf(sx[t * P + pr], Gn[static_cast<int64_t>(pr) * N + n], xg);
                        dh = fmaf(sdy[t * P + pr], Hin[static_cast<int64_t>(pr) * N + n], dh);
                    }
                    dBacc[k] += fmaf(ee, xg, db);
                    dCacc[k] += fmaf(ec, dh, dc);
                }
            }
        }
        __syncthreads();

        // dcs per token, then the decay gradients
        if (tid < kQ) {
            const int t = tid;
            float dcs = 0.f;
            if (t < L) {
                float row = 0.f, col = 0.f;
                for (int s = 0; s <= t; ++s) row += sL[t * kQ + s];
                for (int u = t; u < L; ++u) col += sL[u * kQ + t];
                dcs = row - col + exp2f(scs[t]) * sq1[t] - seend[t] * sq2[t];
                if (t == L - 1) {
                    float hout = exp2f(csend) * gh;
                    for (int s = 0; s < L; ++s) hout = fmaf(seend[s], sq2[s], hout);
                    dcs += hout;
                }
            }
            sdcs[t] = dcs;
        }
        __syncthreads();
        if (tid < kQ) {
            const int k = tid;
            float da = 0.f;
            for (int t = L - 1; t >= k; --t) da += sdcs[t];
            if (k < L) st<T>(p.ddt, (t0 + k) * p.H + h, fmaf(Ah, da, sxdx[k]));
            sq1[k] = k < L ? sdt[k] * da : 0.f;   // dA terms (sq1 is free again)
        }
        __syncthreads();
        if (tid == 0) {
            float sa = 0.f, sd = 0.f;
            for (int k = 0; k < L; ++k) {
                sa += sq1[k];
                sd += sdyx[k];
            }
            p.dAp[bh * p.nC + c] = sa;
            p.dDp[bh * p.nC + c] = sd;
        }
    }

    // this slice's dB and dC for the chunk
    const int t = tt;
    if (t < L) {
        const int64_t base = ((slice * p.b * p.T + t0 + t) * p.G + g) * p.N;
#pragma unroll
        for (int k = 0; k < kMaxNk; ++k) {
            if (k >= nk) break;
            const int n = j + kTpt * k;
            p.dBp[base + n] = dBacc[k];
            p.dCp[base + n] = dCacc[k];
        }
    }
}

// dB, dC = sum over head slices (fixed order), rounded to the input dtype.
template <typename T>
__global__ __launch_bounds__(kThreads) void k_bwd_reduce_bc(BwdParams p)
{
    const int64_t n_el = p.b * p.T * p.G * p.N;
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (i >= n_el) return;
    float sb = 0.f, sc = 0.f;
    for (int64_t s = 0; s < p.S; ++s) {
        sb += p.dBp[s * n_el + i];
        sc += p.dCp[s * n_el + i];
    }
    st<T>(p.dB, i, sb);
    st<T>(p.dC, i, sc);
}

// dA_log[h] = A_h * sum over rows and chunks of the dA terms; dD likewise.
__global__ __launch_bounds__(kThreads) void k_bwd_reduce_head(BwdParams p)
{
    __shared__ float scr[4];
    const int64_t h = blockIdx.x;
    float sa = 0.f, sd = 0.f;
    for (int64_t i = threadIdx.x; i < p.b * p.nC; i += kThreads) {
        const int64_t b = i / p.nC, c = i - b * p.nC;
        sa += p.dAp[(b * p.H + h) * p.nC + c];
        sd += p.dDp[(b * p.H + h) * p.nC + c];
    }
    sa = block_sum256(sa, scr);
    sd = block_sum256(sd, scr);
    if (threadIdx.x == 0) {
        p.dA_log[h] = -expf(p.A_log[h]) * sa;
        if (p.dD) p.dD[h] = sd;
    }
}

template <typename T>
hipError_t launch_all(const BwdParams& p, hipStream_t st, hipEvent_t ev0, hipEvent_t ev1)
{
    const size_t sm_states = sizeof(float) * static_cast<size_t>(kQ) * (2 * p.P + 2 * p.N);
    const size_t sm_chunk = sizeof(float) * (static_cast<size_t>(kQ) * (2 * p.N + 2 * p.P) + 4 * kQ * kQ);
    if (sm_states > 65536) {
        const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_bwd_states<T>),
                                                 hipFuncAttributeMaxDynamicSharedMemorySize,
                                                 static_cast<int>(sm_states));
        if (e != hipSuccess) return e;
    }
    if (sm_chunk > 65536) {
        const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_bwd_chunk<T>),
                                                 hipFuncAttributeMaxDynamicSharedMemorySize,
                                                 static_cast<int>(sm_chunk));
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(k_bwd_states<T>, dim3(static_cast<unsigned>(p.nC), static_cast<unsigned>(p.b),
                                             static_cast<unsigned>(p.H)),
                       dim3(kThreads), sm_states, st, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t nscan = p.b * p.H * p.P * p.N / 4;
    hipLaunchKernelGGL(k_bwd_scan, dim3(static_cast<unsigned>((nscan + kThreads - 1) / kThreads)), dim3(kThreads),
                       0, st, p);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (ev0 && (e = hipEventRecord(ev0, st)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_bwd_chunk<T>, dim3(static_cast<unsigned>(p.nC), static_cast<unsigned>(p.b),
                                            static_cast<unsigned>(p.G * p.S)),
                       dim3(kThreads), sm_chunk, st, p);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (ev1 && (e = hipEventRecord(ev1, st)) != hipSuccess) return e;
    return launch_backward_reduce(p, sizeof(T) == 2, st);
}

template <typename T>
hipError_t launch_reduce(const BwdParams& p, hipStream_t st, bool with_bc)
{
    const int64_t nbc = p.b * p.T * p.G * p.N;
    if (with_bc) {
        hipLaunchKernelGGL(k_bwd_reduce_bc<T>, dim3(static_cast<unsigned>((nbc + kThreads - 1) / kThreads)),
                           dim3(kThreads), 0, st, p);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(k_bwd_reduce_head, dim3(static_cast<unsigned>(p.H)), dim3(kThreads), 0, st, p);
    return hipGetLastError();
}

size_t al(size_t v) { return (v + 255) / 256 * 256; }

}  // namespace

void bwd_slices(int64_t b, int64_t nC, int64_t G, int64_t hpg, int64_t* S, int64_t* hs)
{
    // as few slices as still give every compute unit of the chip (256 CUs) a
    // workgroup: a workgroup shares B, C and the chunk's Gram tiles over its
    // heads and accumulates dB, dC over them (measured at the 2.7B shape:
    // 80 heads per workgroup 1.130 ms, 40: 1.139, 16: 1.165, 8: 1.217)
    constexpr int64_t kCUs = 256;
    const int64_t units = b * nC * G;
    int64_t s = (kCUs + units - 1) / units;
    if (s > hpg) s = hpg;
    if (s < 1) s = 1;
    *hs = (hpg + s - 1) / s;
    *S = (hpg + *hs - 1) / *hs;
}

BwdLayout bwd_layout(int64_t b, int64_t T, int64_t H, int64_t P, int64_t N, int64_t G, int64_t nC, int64_t S,
                     bool fast)
{
    BwdLayout l{};
    size_t off = 0;
    const auto take_bytes = [&](size_t bytes) {
        const size_t o = off;
        off += al(bytes);
        return o;
    };
    const auto take = [&](size_t n) { return take_bytes(n * sizeof(float)); };
    const size_t state_bytes = static_cast<size_t>(b * nC * H * P * N) * (fast ? 2 : 4);
    l.cs = fast ? 0 : take(static_cast<size_t>(b * H * nC * kBwdQ));
    l.hin = take_bytes(state_bytes);
    l.gn = fast ? 0 : take_bytes(state_bytes);
    l.gnT = fast ? take_bytes(state_bytes) : 0;
    l.dBp = take(static_cast<size_t>(S * b * T * G * N));
    l.dCp = take(static_cast<size_t>(S * b * T * G * N));
    l.dAp = take(static_cast<size_t>(b * nC * H));
    l.dDp = take(static_cast<size_t>(b * nC * H));
    l.total = off;
    return l;
}

namespace {

// out[c] = sum over rows r (in order) of part[r][c].
__global__ __launch_bounds__(kThreads) void k_sum_rows(const float* part, int64_t nrows, int64_t ncols, float* out)
{
    const int64_t c = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (c >= ncols) return;
    float s = 0.f;
    for (int64_t r = 0; r < nrows; ++r) s += part[r * ncols + c];
    out[c] = s;
}

}  // namespace

hipError_t launch_sum_rows(const float* part, int64_t nrows, int64_t ncols, float* out, hipStream_t stream)
{
    hipLaunchKernelGGL(k_sum_rows, dim3(static_cast<unsigned>((ncols + kThreads - 1) / kThreads)), dim3(kThreads), 0,
                       stream, part, nrows, ncols, out);
    return hipGetLastError();
}

hipError_t launch_backward_reduce(const BwdParams& p, bool bf16, hipStream_t stream, bool with_bc)
{
    return bf16 ? launch_reduce<uint16_t>(p, stream, with_bc) : launch_reduce<float>(p, stream, with_bc);
}

hipError_t launch_backward(const BwdParams& p, bool bf16, hipStream_t stream, hipEvent_t ev_begin,
                           hipEvent_t ev_end)
{
    return bf16 ? launch_all<uint16_t>(p, stream, ev_begin, ev_end)
                : launch_all<float>(p, stream, ev_begin, ev_end);
}

}  // namespace ssd
