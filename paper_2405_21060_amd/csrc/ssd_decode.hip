// One decode step of the SSD layer: the recurrent (linear-time) form of the
// selective SSM applied to a single new token per sequence (Section 3 / eq. s6
// with scalar A; the per-token inference cost of Section 6.3):
//
//     S <- exp(dt A) S + (dt x) B^T,        y = S C + D x,
//
// per (batch row, head), with S the P x N float32 state, updated in place.
//
// Memory-bound: every step reads and writes the whole state (2 x 4 P N bytes
// per head) and little else.  One thread owns 8 consecutive state columns of
// one state row (p); the N/8 threads of a row are a power-of-two segment of a
// wavefront, so y[p] is a shuffle reduction inside the segment.  State rows are
// read and written as two float4 per thread (fully coalesced, streaming
// stores), B and C of the row's group are read by every row (cache hits).
#include "ssd_device.h"
#include "ssd_internal.h"

namespace ssd {
namespace {

constexpr int kDecodeThreads = 256;

__device__ __forceinline__ float load_act(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float load_act(const uint16_t* p, int64_t i)
{
    return __uint_as_float(static_cast<uint32_t>(p[i]) << 16);
}

__device__ __forceinline__ void store_act(float* p, int64_t i, float v) { p[i] = v; }
__device__ __forceinline__ void store_act(uint16_t* p, int64_t i, float v)
{
    p[i] = __builtin_bit_cast(uint16_t, static_cast<__bf16>(v));   // round to nearest even
}

// seg = threads per state row (power of two, >= N/8, <= 32)
template <typename T>
__global__ __launch_bounds__(kDecodeThreads) void k_decode_step(DecodeParams p, int seg, int log2seg)
{
    const int64_t rows = p.b * p.H * p.P;
    const int rows_per_block = kDecodeThreads / seg;
    const int lane_in_row = threadIdx.x & (seg - 1);
    const int64_t row = static_cast<int64_t>(blockIdx.x) * rows_per_block + (threadIdx.x >> log2seg);
    const int n0 = 8 * lane_in_row;
    const bool active = row < rows && n0 < p.N;
    const T* x = static_cast<const T*>(p.x);
    const T* dt = static_cast<const T*>(p.dt);
    const T* Bm = static_cast<const T*>(p.B);
    const T* Cm = static_cast<const T*>(p.C);
    float ysum = 0.f, xv = 0.f, Dh = 0.f;
    if (active) {
        const int64_t bh = row / p.P;             // (batch row, head)
        const int64_t b = bh / p.H, h = bh - b * p.H;
        const int64_t g = h / (p.H / p.G);
        const float dtv = load_act(dt, bh);
        const float dA = expf(dtv * -expf(p.A_log[h]));
        xv = load_act(x, row);
        Dh = p.D ? p.D[h] : 0.f;
        const float u = dtv * xv;
        float4* sp = reinterpret_cast<float4*>(p.state + row * p.N + n0);
        const float4 s0 = sp[0], s1 = sp[1];
        const int64_t bg = (b * p.G + g) * p.N + n0;
        float bv[8], cv[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            bv[e] = load_act(Bm, bg + e);
            cv[e] = load_act(Cm, bg + e);
        }
        const float sv[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
        float ns[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            ns[e] = dA * sv[e] + u * bv[e];
            ysum += ns[e] * cv[e];
        }
        typedef float f4 __attribute__((ext_vector_type(4)));
        __builtin_nontemporal_store(f4{ns[0], ns[1], ns[2], ns[3]}, reinterpret_cast<f4*>(sp));
        __builtin_nontemporal_store(f4{ns[4], ns[5], ns[6], ns[7]}, reinterpret_cast<f4*>(sp + 1));
    }
    for (int off = seg >> 1; off > 0; off >>= 1) ysum += __shfl_xor(ysum, off, 64);
    if (active && lane_in_row == 0) store_act(static_cast<T*>(p.y), row, ysum + Dh * xv);
}

}  // namespace

hipError_t launch_decode(const DecodeParams& p, bool bf16, hipStream_t stream)
{
    int seg = 1, log2seg = 0;
    while (seg < p.N / 8) {
        seg <<= 1;
        ++log2seg;
    }
    const int64_t rows = p.b * p.H * p.P;
    const int64_t rows_per_block = kDecodeThreads / seg;
    const unsigned grid = static_cast<unsigned>((rows + rows_per_block - 1) / rows_per_block);
    if (bf16)
        hipLaunchKernelGGL(k_decode_step<uint16_t>, dim3(grid), dim3(kDecodeThreads), 0, stream, p, seg, log2seg);
    else
        hipLaunchKernelGGL(k_decode_step<float>, dim3(grid), dim3(kDecodeThreads), 0, stream, p, seg, log2seg);
    return hipGetLastError();
}

}  // namespace ssd
