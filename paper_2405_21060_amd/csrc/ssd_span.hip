// A sequence split into consecutive spans (context parallelism, Section 8.2):
// each span runs the layer from a zero state (ssd_forward); these kernels do
// the rest of the state passing on one GPU's span.
//
//   k_span_decay     total decay of the span per (batch, head):
//                    exp(A_h sum_t dt_t).
//   k_span_combine   exclusive scan over spans of (decay, state) pairs under
//                    the scalar-SSM operator of Appendix B,
//                    (a, h) then (a', h')  =  (a a', a' h + h'):
//                    the state entering every span, and the final state.
//   k_chunk_dt_sums, k_span_correct
//                    the output a span's entering state h_in adds:
//                    y_t += exp(A_h sum_{s<=t} dt_s) (h_in C_t),
//                    a dense (P x N) x (N x tokens) product per (batch, head)
//                    on the matrix cores for bf16, with the decay of every
//                    token from a chunk-level prefix of dt sums.
#include "ssd_device.h"
#include "ssd_internal.h"

namespace ssd {
namespace {

constexpr int kSpanThreads = 256;
constexpr int kSpanQ = 256;          // tokens per workgroup of the correction
constexpr int kMaxPT = 8;            // 16-row p-tiles of the largest head dimension (128)

template <typename T>
__device__ __forceinline__ float ld_act(const T* p, int64_t i) { return Act<T>::load(p, i); }

// Sum of `v` over the 256 threads of the block, in a fixed order.
__device__ __forceinline__ float block_sum(float v, float* scratch)
{
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) scratch[w] = v;
    __syncthreads();
    const float s = (scratch[0] + scratch[1]) + (scratch[2] + scratch[3]);
    __syncthreads();
    return s;
}

template <typename T>
__global__ __launch_bounds__(kSpanThreads) void k_span_decay(int64_t T_, int64_t H, const T* dt,
                                                             const float* A_log, float* decay)
{
    __shared__ float scr[kSpanThreads / 64];
    const int64_t bh = blockIdx.x;
    const int64_t b = bh / H, h = bh - b * H;
    float s = 0.f;
    for (int64_t t = threadIdx.x; t < T_; t += kSpanThreads) s += ld_act(dt, (b * T_ + t) * H + h);
    s = block_sum(s, scr);
    if (threadIdx.x == 0) decay[bh] = expf(-expf(A_log[h]) * s);
}

// One thread per 4 consecutive state elements of one (batch, head).
__global__ __launch_bounds__(kSpanThreads) void k_span_combine(int64_t R, int64_t bh_count, int64_t PN,
                                                               const float* decay, const float* local,
                                                               const float* init, float* entering,
                                                               float* fin)
{
    const int64_t q = static_cast<int64_t>(blockIdx.x) * kSpanThreads + threadIdx.x;   // float4 index
    const int64_t per = bh_count * PN;   // elements of one span's states
    if (4 * q >= per) return;
    const int64_t bh = (4 * q) / PN;
    float4 acc = init ? reinterpret_cast<const float4*>(init)[q] : make_float4(0.f, 0.f, 0.f, 0.f);
    for (int64_t r = 0; r < R; ++r) {
        reinterpret_cast<float4*>(entering + r * per)[q] = acc;
        const float a = decay[r * bh_count + bh];
        const float4 l = reinterpret_cast<const float4*>(local + r * per)[q];
        acc = make_float4(a * acc.x + l.x, a * acc.y + l.y, a * acc.z + l.z, a * acc.w + l.w);
    }
    if (fin) reinterpret_cast<float4*>(fin)[q] = acc;
}

// dt sums of every 256-token chunk of the span, per (batch, head).
template <typename T>
__global__ __launch_bounds__(kSpanThreads) void k_chunk_dt_sums(SpanParams p)
{
    __shared__ float scr[kSpanThreads / 64];
    const int c = blockIdx.x;
    const int64_t bh = blockIdx.y;
    const int64_t b = bh / p.H, h = bh - b * p.H;
    const int64_t t = static_cast<int64_t>(c) * kSpanQ + threadIdx.x;
    float v = t < p.T ? ld_act(static_cast<const T*>(p.dt), (b * p.T + t) * p.H + h) : 0.f;
    v = block_sum(v, scr);
    if (threadIdx.x == 0) p.sums[bh * p.nC + c] = v;
}

// Per-token decay factors of a chunk into LDS: exp2(log2e A (sum of dt over
// the span up to and including the token)), every factor <= 1.
template <typename T>
__device__ __forceinline__ void chunk_decays(const SpanParams& p, int c, int64_t b, int64_t h, int L,
                                             float* ev, float* scr)
{
    const float A2 = -expf(p.A_log[h]) * kLog2e;
    // sum of the chunk sums before this chunk (at most nC of them)
    float pre = 0.f;
    for (int k = threadIdx.x; k < c; k += kSpanThreads) pre += p.sums[(b * p.H + h) * p.nC + k];
    pre = block_sum(pre, scr);
    const int t = threadIdx.x;
    float a = t < L ? ld_act(static_cast<const T*>(p.dt), (b * p.T + static_cast<int64_t>(c) * kSpanQ + t) * p.H + h) : 0.f;
    // inclusive scan: wavefront shuffles, then the wavefront totals
    const int lane = t & 63, w = t >> 6;
    for (int sh = 1; sh < 64; sh <<= 1) {
        const float o = __shfl_up(a, sh, 64);
        if (lane >= sh) a += o;
    }
    if (lane == 63) scr[w] = a;
    __syncthreads();
    float before = 0.f;
    for (int k = 0; k < w; ++k) before += scr[k];
    ev[t] = t < L ? exp2f(A2 * (pre + before + a)) : 0.f;
    __syncthreads();
}

// bf16: matrix cores.  Wavefront w takes tokens 64 w .. 64 w + 63 (four
// 16-token strips); per strip and 16-row p-tile, Y^T[p][t] = sum_n E[p][n] C[t][n]
// over K-steps of 32 (v_mfma_f32_16x16x32_bf16: E rows from LDS as the A
// operand, C rows of the strip's tokens straight from memory as the B
// operand), then y[t][p] += decay_t Y^T[p][t].  KN = K-steps (N padded to 32):
// the K loop is unrolled at compile time, so that the accumulator reads after
// the last matrix-core instruction get their wait states on every path.
template <int KN>
__global__ __launch_bounds__(kSpanThreads) void k_span_correct_bf16(SpanParams p)
{
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    float* ev = reinterpret_cast<float*>(smem);                       // kSpanQ
    float* scr = ev + kSpanQ;                                           // 4
    constexpr int NP = 32 * KN;                                         // N padded to the K-step
    const int ES = NP + 8;                                              // LDS row stride (bf16)
    uint16_t* E = reinterpret_cast<uint16_t*>(scr + 4);                 // P x ES

    const int c = blockIdx.x;
    const int64_t bh = blockIdx.y;
    const int64_t b = bh / p.H, h = bh - b * p.H;
    const int64_t g = h / (p.H / p.G);
    const int64_t t0 = static_cast<int64_t>(c) * kSpanQ;
    const int L = static_cast<int>(kSpanQ < p.T - t0 ? kSpanQ : p.T - t0);
    const int P = static_cast<int>(p.P), N = static_cast<int>(p.N);

    // the entering state, rounded to bf16 (zero-padded columns up to NP): float4
    // loads, 8-byte LDS stores
    const float4* Eg4 = reinterpret_cast<const float4*>(p.entering + bh * p.P * p.N);
    const int quads = P * N / 4, qrow = N / 4;
#pragma unroll 8
    for (int i = threadIdx.x; i < quads; i += kSpanThreads) {
        const float4 f = Eg4[i];
        const int pr = i / qrow, n = 4 * (i - pr * qrow);
        const float fv[4] = {f.x, f.y, f.z, f.w};
        uint32_t hv[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {   // round to nearest even
            const uint32_t u = __float_as_uint(fv[e]);
            hv[e] = (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
        }
        *reinterpret_cast<uint2*>(E + pr * ES + n) = make_uint2(hv[0] | (hv[1] << 16), hv[2] | (hv[3] << 16));
    }
    if (NP > N)
        for (int i = threadIdx.x; i < P * (NP - N); i += kSpanThreads) {
            const int pr = i / (NP - N);
            E[pr * ES + N + (i - pr * (NP - N))] = 0;
        }
    chunk_decays<uint16_t>(p, c, b, h, L, ev, scr);   // ends with a barrier

    const int lane = threadIdx.x & 63, r = lane & 15, lg = lane >> 4;
    const int w = threadIdx.x >> 6;
    const uint16_t* Cb = static_cast<const uint16_t*>(p.C);
    uint16_t* y = static_cast<uint16_t*>(p.y);
    for (int s = 0; s < 4; ++s) {
        const int tl = 64 * w + 16 * s + r;                      // this lane's token (B column)
        if (16 * (4 * w + s) >= L) break;                        // strip entirely past the span's end
        const int tc = tl < L ? tl : L - 1;
        const uint16_t* crow = Cb + ((b * p.T + t0 + tc) * p.G + g) * p.N;
        // the strip's C fragments (shared by every p-tile) and the y values the
        // lane updates, requested together
        uint4 cf[KN];
#pragma unroll
        for (int k = 0; k < KN; ++k) {
            const int n0 = 32 * k + 8 * lg;
            cf[k] = n0 < N ? *reinterpret_cast<const uint4*>(crow + n0) : make_uint4(0, 0, 0, 0);
        }
        const int64_t yrow = ((b * p.T + t0 + tc) * p.H + h) * p.P + 4 * lg;
        uint2 yo[kMaxPT];
#pragma unroll
        for (int pt = 0; pt < kMaxPT; ++pt)
            if (pt < P / 16) yo[pt] = *reinterpret_cast<const uint2*>(y + yrow + 16 * pt);
        const float e = ev[tl];
#pragma unroll
        for (int pt = 0; pt < kMaxPT; ++pt) {
            if (pt >= P / 16) break;
            f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int k = 0; k < KN; ++k) {
                const uint4 av = *reinterpret_cast<const uint4*>(E + (16 * pt + r) * ES + 32 * k + 8 * lg);
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, av),
                                                              __builtin_bit_cast(bf16x8_t, cf[k]), acc, 0, 0, 0);
            }
            if (tl < L) {
                const uint2 o = yo[pt];
                const float yv[4] = {__uint_as_float(o.x << 16), __uint_as_float(o.x & 0xFFFF0000u),
                                     __uint_as_float(o.y << 16), __uint_as_float(o.y & 0xFFFF0000u)};
                uint16_t* dst = y + yrow + 16 * pt;
#pragma unroll
                for (int v = 0; v < 4; ++v) Act<uint16_t>::store(dst, v, yv[v] + e * acc[v]);
            }
        }
    }
}

// float32: plain FMAs (the matrix-core path rounds its operands to bf16).
// Thread t handles token t of the chunk; E is read by every thread alike.
__global__ __launch_bounds__(kSpanThreads) void k_span_correct_f32(SpanParams p)
{
    __shared__ float ev[kSpanQ];
    __shared__ float scr[kSpanThreads / 64];
    const int c = blockIdx.x;
    const int64_t bh = blockIdx.y;
    const int64_t b = bh / p.H, h = bh - b * p.H;
    const int64_t g = h / (p.H / p.G);
    const int64_t t0 = static_cast<int64_t>(c) * kSpanQ;
    const int L = static_cast<int>(kSpanQ < p.T - t0 ? kSpanQ : p.T - t0);
    chunk_decays<float>(p, c, b, h, L, ev, scr);
    const int t = threadIdx.x;
    if (t >= L) return;
    const float* Eg = p.entering + bh * p.P * p.N;
    const float* crow = static_cast<const float*>(p.C) + ((b * p.T + t0 + t) * p.G + g) * p.N;
    float* y = static_cast<float*>(p.y) + ((b * p.T + t0 + t) * p.H + h) * p.P;
    const float e = ev[t];
    for (int64_t pr = 0; pr < p.P; ++pr) {
        float acc = 0.f;
        for (int64_t n = 0; n < p.N; ++n) acc += Eg[pr * p.N + n] * crow[n];
        y[pr] += e * acc;
    }
}

}  // namespace

hipError_t launch_span_decay(int64_t b, int64_t T, int64_t H, const void* dt, const float* A_log, float* decay,
                             bool bf16, hipStream_t stream)
{
    const dim3 grid(static_cast<unsigned>(b * H));
    if (bf16)
        hipLaunchKernelGGL(k_span_decay<uint16_t>, grid, dim3(kSpanThreads), 0, stream, T, H,
                           static_cast<const uint16_t*>(dt), A_log, decay);
    else
        hipLaunchKernelGGL(k_span_decay<float>, grid, dim3(kSpanThreads), 0, stream, T, H,
                           static_cast<const float*>(dt), A_log, decay);
    return hipGetLastError();
}

hipError_t launch_span_combine(int64_t R, int64_t bh, int64_t PN, const float* decay, const float* local,
                               const float* init, float* entering, float* fin, hipStream_t stream)
{
    const int64_t quads = bh * PN / 4;
    const dim3 grid(static_cast<unsigned>((quads + kSpanThreads - 1) / kSpanThreads));
    hipLaunchKernelGGL(k_span_combine, grid, dim3(kSpanThreads), 0, stream, R, bh, PN, decay, local, init,
                       entering, fin);
    return hipGetLastError();
}

int64_t span_chunks(int64_t T) { return (T + kSpanQ - 1) / kSpanQ; }

hipError_t launch_span_correct(const SpanParams& p, bool bf16, hipStream_t stream)
{
    const dim3 grid(static_cast<unsigned>(p.nC), static_cast<unsigned>(p.b * p.H));
    if (bf16) {
        hipLaunchKernelGGL(k_chunk_dt_sums<uint16_t>, grid, dim3(kSpanThreads), 0, stream, p);
        const int KN = static_cast<int>((p.N + 31) / 32);
        const size_t lds = sizeof(float) * (kSpanQ + 4) + sizeof(uint16_t) * static_cast<size_t>(p.P * (32 * KN + 8));
        auto go = [&](auto kern) -> hipError_t {
            if (lds > 64 * 1024) {   // up to 68 KB (P 128, N 256): above the default dynamic-LDS limit
                const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                                         hipFuncAttributeMaxDynamicSharedMemorySize,
                                                         static_cast<int>(lds));
                if (e != hipSuccess) return e;
            }
            hipLaunchKernelGGL(kern, grid, dim3(kSpanThreads), lds, stream, p);
            return hipSuccess;
        };
        hipError_t e = hipSuccess;
        switch (KN) {
        case 1: e = go(k_span_correct_bf16<1>); break;
        case 2: e = go(k_span_correct_bf16<2>); break;
        case 3: e = go(k_span_correct_bf16<3>); break;
        case 4: e = go(k_span_correct_bf16<4>); break;
        case 5: e = go(k_span_correct_bf16<5>); break;
        case 6: e = go(k_span_correct_bf16<6>); break;
        case 7: e = go(k_span_correct_bf16<7>); break;
        default: e = go(k_span_correct_bf16<8>); break;   // N <= 256
        }
        if (e != hipSuccess) return e;
    } else {
        hipLaunchKernelGGL(k_chunk_dt_sums<float>, grid, dim3(kSpanThreads), 0, stream, p);
        hipLaunchKernelGGL(k_span_correct_f32, grid, dim3(kSpanThreads), 0, stream, p);
    }
    return hipGetLastError();
}

}  // namespace ssd
