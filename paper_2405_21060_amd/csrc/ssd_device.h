// Device-side building blocks shared by the SSD kernels (gfx950 / CDNA4).
//
// Matrix-core convention used throughout.  A 16x16 output tile is produced by
// "K-steps" of 32 contraction indices.  In a K-step every lane l holds eight
// values of each operand: lane row/column r = l & 15, lane group g = l >> 4,
// slot e = 0..7 carries contraction index k = kmap(g, e).  The A operand's
// lane holds row r (A[r][k]), the B operand's lane holds column r (B[k][r]).
// Any kmap that is a bijection onto the 32 indices gives the same sum, because
// both operands use the same lane/slot -> k assignment.
//   * bf16: one v_mfma_f32_16x16x32_bf16 (slot e of group g is one of its k);
//   * f32 : eight v_mfma_f32_16x16x4_f32, instruction e contracting the four
//           values {slot e of group 0..3}.
// The accumulator (4 floats per lane) holds D[4 g + v][r], v = 0..3.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ssd {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;

struct Frag8 {
    float v[8];
};

// Activation element access: float, or bfloat16 stored as its 16 bits.
template <typename T>
struct Act;

// The block path's dt: softplus(v) = max(v, 0) + log(1 + e^-|v|) (no overflow
// on either side), after the head's bias, then the clamp.
__device__ __forceinline__ float softplus_f(float v) { return fmaxf(v, 0.f) + log1pf(expf(-fabsf(v))); }

template <>
struct Act<float> {
    static __device__ __forceinline__ float load(const float* p, int64_t i) { return p[i]; }
    static __device__ __forceinline__ void store(float* p, int64_t i, float v) { p[i] = v; }
};

template <>
struct Act<uint16_t> {
    static __device__ __forceinline__ float load(const uint16_t* p, int64_t i)
    {
        return __uint_as_float(static_cast<uint32_t>(p[i]) << 16);
    }
    // round to nearest even (inputs are finite)
    static __device__ __forceinline__ void store(uint16_t* p, int64_t i, float v)
    {
        uint32_t u = __float_as_uint(v);
        u += 0x7FFFu + ((u >> 16) & 1u);
        p[i] = static_cast<uint16_t>(u >> 16);
    }
};

__device__ __forceinline__ f32x4_t mma_step(const Frag8& a, const Frag8& b, f32x4_t c, uint16_t)
{
    bf16x8_t av, bv;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        av[e] = static_cast<__bf16>(a.v[e]);
        bv[e] = static_cast<__bf16>(b.v[e]);
    }
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, c, 0, 0, 0);
}

__device__ __forceinline__ f32x4_t mma_step(const Frag8& a, const Frag8& b, f32x4_t c, float)
{
#pragma unroll
    for (int e = 0; e < 8; ++e)
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[e], b.v[e], c, 0, 0, 0);
    return c;
}

__device__ __forceinline__ f32x4_t zero4()
{
    f32x4_t z = {0.f, 0.f, 0.f, 0.f};
    return z;
}

// Inclusive prefix sum over the first `nthreads` (a multiple of 64, <= 1024)
// threads of the block; `scratch` holds nthreads/64 floats of shared memory.
__device__ __forceinline__ float block_inclusive_scan(float v, float* scratch)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        float o = __shfl_up(v, d, 64);
        if (lane >= d) v += o;
    }
    if (lane == 63) scratch[wave] = v;
    __syncthreads();
    float off = 0.f;
    for (int w = 0; w < wave; ++w) off += scratch[w];
    __syncthreads();
    return v + off;
}

}  // namespace ssd
