// Output side of the Mamba-2 block around the SSD layer, as one pass over y:
// the gate y * SiLU(z) of the block equations of Section 8.1 and the grouped
// RMS normalisation placed after it (Section 7.1), per token row of H * P
// channels (head-major), in place.  Used by the general path, and by the fused
// path for normalisation groups wider than one head (the fused chunk kernel
// gates, and normalises single-head groups, in its own output stage).
//
// Memory-bound: each element of y (and z) is read once; a lane keeps its
// gated pieces in registers between the group's sum of squares and the scaled
// store (groups too wide for that read them a second time, from cache).  A group of
// `group` channels is `group / 8` pieces of 8 channels (one 16- or 32-byte
// vector); `seg` lanes (a power of two, at most 64) share a group and reduce
// its sum with shuffles inside their segment; a wavefront holds 64 / seg groups.
#include "ssd_device.h"
#include "ssd_internal.h"

namespace ssd {
namespace {

constexpr int kGateNormThreads = 256;

template <typename T>
struct Vec8;

template <>
struct Vec8<uint16_t> {
    static __device__ __forceinline__ void load(const uint16_t* p, int64_t i, float* v)
    {
        const uint4 u = *reinterpret_cast<const uint4*>(p + i);
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            v[2 * k] = __uint_as_float(w[k] << 16);
            v[2 * k + 1] = __uint_as_float(w[k] & 0xFFFF0000u);
        }
    }
    static __device__ __forceinline__ void store(uint16_t* p, int64_t i, const float* v)
    {
        uint32_t w[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
            bf16x2_t h;
            h[0] = static_cast<__bf16>(v[2 * k]);       // round to nearest even
            h[1] = static_cast<__bf16>(v[2 * k + 1]);
            w[k] = __builtin_bit_cast(uint32_t, h);
        }
        *reinterpret_cast<uint4*>(p + i) = make_uint4(w[0], w[1], w[2], w[3]);
    }
};

template <>
struct Vec8<float> {
    static __device__ __forceinline__ void load(const float* p, int64_t i, float* v)
    {
        const float4 a = *reinterpret_cast<const float4*>(p + i);
        const float4 b = *reinterpret_cast<const float4*>(p + i + 4);
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
        v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    }
    static __device__ __forceinline__ void store(float* p, int64_t i, const float* v)
    {
        *reinterpret_cast<float4*>(p + i) = make_float4(v[0], v[1], v[2], v[3]);
        *reinterpret_cast<float4*>(p + i + 4) = make_float4(v[4], v[5], v[6], v[7]);
    }
};

__device__ __forceinline__ float silu_f(float z) { return z / (1.f + expf(-z)); }

// Gated piece: y, times SiLU(z) when gating.
template <typename T>
__device__ __forceinline__ void gated_piece(const GateNormParams& p, int64_t e, float* g)
{
    Vec8<T>::load(static_cast<const T*>(p.y), e, g);
    if (p.z) {
        float zv[8];
        Vec8<T>::load(static_cast<const T*>(p.z), e, zv);
#pragma unroll
        for (int k = 0; k < 8; ++k) g[k] *= silu_f(zv[k]);
    }
}

// Gate only: one piece per thread.
template <typename T>
__global__ __launch_bounds__(kGateNormThreads) void k_gate(GateNormParams p)
{
    const int64_t pieces = p.rows * (p.C / 8);
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kGateNormThreads + threadIdx.x;
    if (i >= pieces) return;
    float g[8];
    gated_piece<T>(p, 8 * i, g);
    Vec8<T>::store(static_cast<T*>(p.y), 8 * i, g);
}

// Gate (optional) and grouped RMS normalisation.  Each lane keeps its (at most
// MAXP) gated pieces of the group in registers between the sum of squares and
// the scaled store; groups with more pieces per lane than MAXP (MAXP == 0)
// re-read them instead.
template <typename T, int MAXP>
__global__ __launch_bounds__(kGateNormThreads) void k_gate_norm(GateNormParams p, int seg, int log2seg)
{
    const int lane = threadIdx.x & 63;
    const int per_wave = 64 >> log2seg;
    const int64_t groups_per_row = p.C / p.group;
    const int64_t ngroups = p.rows * groups_per_row;
    const int64_t gid = (static_cast<int64_t>(blockIdx.x) * (kGateNormThreads / 64) + (threadIdx.x >> 6)) * per_wave +
                        (lane >> log2seg);
    const int li = lane & (seg - 1);
    const bool active = gid < ngroups;
    const int64_t row = active ? gid / groups_per_row : 0;
    const int64_t c0 = active ? (gid - row * groups_per_row) * p.group : 0;
    const int64_t base = row * p.C + c0;
    const int pieces = static_cast<int>(p.group / 8);
    float ss = 0.f;
    float g[MAXP > 0 ? MAXP : 1][8];
    if (active) {
        if constexpr (MAXP > 0) {
#pragma unroll
            for (int k = 0; k < MAXP; ++k)
                if (li + k * seg < pieces) gated_piece<T>(p, base + 8 * (li + k * seg), g[k]);
#pragma unroll
            for (int k = 0; k < MAXP; ++k)
                if (li + k * seg < pieces)
#pragma unroll
                    for (int e = 0; e < 8; ++e) ss += g[k][e] * g[k][e];
        } else {
            for (int j = li; j < pieces; j += seg) {
                gated_piece<T>(p, base + 8 * j, g[0]);
#pragma unroll
                for (int e = 0; e < 8; ++e) ss += g[0][e] * g[0][e];
            }
        }
    }
    // sum over the segment's lanes (same fixed tree for every group: deterministic)
    for (int off = seg >> 1; off > 0; off >>= 1) ss += __shfl_xor(ss, off, 64);
    if (!active) return;
    const float scale = 1.f / sqrtf(ss / static_cast<float>(p.group) + p.eps);
    auto finish = [&](int j, float* v) {
        if (p.weight) {
            const float4 w0 = *reinterpret_cast<const float4*>(p.weight + c0 + 8 * j);
            const float4 w1 = *reinterpret_cast<const float4*>(p.weight + c0 + 8 * j + 4);
            const float wv[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = v[e] * scale * wv[e];
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] *= scale;
        }
        Vec8<T>::store(static_cast<T*>(p.y), base + 8 * j, v);
    };
    if constexpr (MAXP > 0) {
#pragma unroll
        for (int k = 0; k < MAXP; ++k)
            if (li + k * seg < pieces) finish(li + k * seg, g[k]);
    } else {
        for (int j = li; j < pieces; j += seg) {
            gated_piece<T>(p, base + 8 * j, g[0]);
            finish(j, g[0]);
        }
    }
}

}  // namespace

hipError_t launch_gate_norm(const GateNormParams& p, bool bf16, hipStream_t stream)
{
    if (p.group == 0) {
        if (!p.z) return hipSuccess;
        const int64_t pieces = p.rows * (p.C / 8);
        const unsigned grid = static_cast<unsigned>((pieces + kGateNormThreads - 1) / kGateNormThreads);
        if (bf16)
            hipLaunchKernelGGL(k_gate<uint16_t>, dim3(grid), dim3(kGateNormThreads), 0, stream, p);
        else
            hipLaunchKernelGGL(k_gate<float>, dim3(grid), dim3(kGateNormThreads), 0, stream, p);
        return hipGetLastError();
    }
    const int64_t pieces = p.group / 8;
    int seg = 1, log2seg = 0;
    while (seg < pieces && seg < 64) {
        seg <<= 1;
        ++log2seg;
    }
    const int64_t ngroups = p.rows * (p.C / p.group);
    const int64_t per_block = (kGateNormThreads / 64) * (64 / seg);
    const unsigned grid = static_cast<unsigned>((ngroups + per_block - 1) / per_block);
    const int64_t per_lane = (pieces + seg - 1) / seg;
    auto go = [&](auto kern) {
        hipLaunchKernelGGL(kern, dim3(grid), dim3(kGateNormThreads), 0, stream, p, seg, log2seg);
    };
    if (bf16) {
        if (per_lane <= 1) go(k_gate_norm<uint16_t, 1>);
        else if (per_lane <= 2) go(k_gate_norm<uint16_t, 2>);
        else if (per_lane <= 4) go(k_gate_norm<uint16_t, 4>);
        else if (per_lane <= 16) go(k_gate_norm<uint16_t, 16>);
        else go(k_gate_norm<uint16_t, 0>);
    } else {
        if (per_lane <= 1) go(k_gate_norm<float, 1>);
        else if (per_lane <= 2) go(k_gate_norm<float, 2>);
        else if (per_lane <= 4) go(k_gate_norm<float, 4>);
        else if (per_lane <= 16) go(k_gate_norm<float, 16>);
        else go(k_gate_norm<float, 0>);
    }
    return hipGetLastError();
}

}  // namespace ssd
