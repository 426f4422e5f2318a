// Gradients of the block steps around the SSD layer (the forward is
// ssd_forward_block: dt parameterisation, the layer, the SiLU gate of the
// block equations of Section 8.1, the grouped RMS normalisation of Section
// 7.1).  The paper gives no backward; these are the chain rule through each
// step, in reverse:
//
//   norm  r = sqrt(mean_group(g^2) + eps), n = g / r, out = n w:
//         dn = dout w,  dg = (dn - n mean_group(dn n)) / r,  dw = sum_rows dout n
//   gate  g = y SiLU(z):  dy = dg SiLU(z),  dz = dg y SiLU'(z),
//         SiLU'(z) = s (1 + z (1 - s)), s = sigmoid(z)
//   dt    dt = clamp(softplus(dt_raw + bias), lo, hi):
//         d dt_raw = ddt [lo < softplus < hi] sigmoid(dt_raw + bias),
//         d bias = sum_rows d dt_raw
//
// The layer's own gradient in between is ssd_backward.  Sums over rows go
// through per-chunk partials and a fixed-order sum (deterministic).
#include "ssd_block_bwd.h"
#include "ssd_device.h"

namespace ssd {
namespace {

constexpr int kBT = 256;

template <typename T>
__device__ __forceinline__ float ldv(const void* p, int64_t i) { return Act<T>::load(static_cast<const T*>(p), i); }

template <typename T>
__device__ __forceinline__ void stv(void* p, int64_t i, float v) { Act<T>::store(static_cast<T*>(p), i, v); }

__device__ __forceinline__ float sigmoid_f(float v)
{
    const float e = expf(-fabsf(v));
    return v >= 0.f ? 1.f / (1.f + e) : e / (1.f + e);
}

// The dt step of the forward, into a buffer of the activation dtype.
template <typename T>
__global__ __launch_bounds__(kBT) void k_dt_apply(BlockBwdParams p)
{
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kBT + threadIdx.x;
    if (i >= p.rows * p.H) return;
    const int64_t h = i % p.H;
    float v = ldv<T>(p.dt_raw, i) + (p.bias ? p.bias[h] : 0.f);
    if (p.softplus) v = softplus_f(v);
    stv<T>(p.dt, i, fminf(fmaxf(v, p.lo), p.hi));
}

// d dt_raw, and per-chunk partial sums over rows for d bias.  Thread = head,
// block (x, y) = (heads, chunk of kRowsPerChunk rows).
constexpr int kRowsPerChunk = 64;

template <typename T>
__global__ __launch_bounds__(kBT) void k_dt_bwd(BlockBwdParams p)
{
    const int64_t h = static_cast<int64_t>(blockIdx.x) * kBT + threadIdx.x;
    if (h >= p.H) return;
    const int64_t r0 = static_cast<int64_t>(blockIdx.y) * kRowsPerChunk;
    const int64_t r1 = r0 + kRowsPerChunk < p.rows ? r0 + kRowsPerChunk : p.rows;
    const float bias = p.bias ? p.bias[h] : 0.f;
    float acc = 0.f;
    for (int64_t r = r0; r < r1; ++r) {
        const int64_t i = r * p.H + h;
        const float v = ldv<T>(p.dt_raw, i) + bias;
        const float sp = p.softplus ? softplus_f(v) : v;
        const bool in = sp > p.lo && sp < p.hi;
        const float dv = in ? ldv<T>(p.ddt, i) * (p.softplus ? sigmoid_f(v) : 1.f) : 0.f;
        stv<T>(p.ddt_raw, i, dv);
        acc += dv;
    }
    if (p.dbias_part) p.dbias_part[blockIdx.y * p.H + h] = acc;
}

// Gate only: dy = dout SiLU(z), dz = dout y SiLU'(z), elementwise.
template <typename T>
__global__ __launch_bounds__(kBT) void k_gate_bwd(BlockBwdParams p)
{
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kBT + threadIdx.x;
    if (i >= p.rows * p.C) return;
    const float z = ldv<T>(p.z, i), s = sigmoid_f(z), d = ldv<T>(p.dout, i);
    stv<T>(p.dy, i, d * z * s);
    stv<T>(p.dz, i, d * ldv<T>(p.y, i) * s * (1.f + z * (1.f - s)));
}

// Gated value of channel i: y SiLU(z) (or y).
template <typename T>
__device__ __forceinline__ float gated(const BlockBwdParams& p, int64_t i, float* zv, float* yv)
{
    const float y = ldv<T>(p.y, i);
    *yv = y;
    if (!p.z) return y;
    const float z = ldv<T>(p.z, i);
    *zv = z;
    return y * z * sigmoid_f(z);
}

// Normalisation (after the optional gate), one group of `group` channels per
// `seg` lanes (a power of two, at most 64): three passes over the group's
// channels (sum of squares; sum of dn n; the gradients), the sums reduced
// inside the segment by a fixed shuffle tree.  Also records 1 / r per (row,
// group) for the weight gradient.
template <typename T>
__global__ __launch_bounds__(kBT) void k_norm_bwd(BlockBwdParams p, int seg, int log2seg)
{
    const int lane = threadIdx.x & 63;
    const int per_wave = 64 >> log2seg;
    const int64_t gpr = p.C / p.group;
    const int64_t ngroups = p.rows * gpr;
    const int64_t gid = (static_cast<int64_t>(blockIdx.x) * (kBT / 64) + (threadIdx.x >> 6)) * per_wave +
                        (lane >> log2seg);
    const int li = lane & (seg - 1);
    const bool active = gid < ngroups;
    const int64_t row = active ? gid / gpr : 0;
    const int64_t c0 = active ? (gid - row * gpr) * p.group : 0;
    const int64_t base = row * p.C + c0;
    float zv = 0.f, yv = 0.f;
    float ss = 0.f;
    if (active)
        for (int64_t j = li; j < p.group; j += seg) {
            const float g = gated<T>(p, base + j, &zv, &yv);
            ss += g * g;
        }
    for (int off = seg >> 1; off > 0; off >>= 1) ss += __shfl_xor(ss, off, 64);
    const float inv = 1.f / sqrtf(ss / static_cast<float>(p.group) + p.eps);
    float sdn = 0.f;
    if (active)
        for (int64_t j = li; j < p.group; j += seg) {
            const float n = gated<T>(p, base + j, &zv, &yv) * inv;
            const float dn = ldv<T>(p.dout, base + j) * (p.w ? p.w[c0 + j] : 1.f);
            sdn += dn * n;
        }
    for (int off = seg >> 1; off > 0; off >>= 1) sdn += __shfl_xor(sdn, off, 64);
    if (!active) return;
    const float mdn = sdn / static_cast<float>(p.group);
    for (int64_t j = li; j < p.group; j += seg) {
        const float n = gated<T>(p, base + j, &zv, &yv) * inv;
        const float dn = ldv<T>(p.dout, base + j) * (p.w ? p.w[c0 + j] : 1.f);
        const float dg = (dn - n * mdn) * inv;
        if (p.z) {
            const float s = sigmoid_f(zv);
            stv<T>(p.dy, base + j, dg * zv * s);
            stv<T>(p.dz, base + j, dg * yv * s * (1.f + zv * (1.f - s)));
        } else {
            stv<T>(p.dy, base + j, dg);
        }
    }
    if (li == 0 && p.inv_rms) p.inv_rms[gid] = inv;
}

// Per-chunk partial sums over rows of dout n for the weight gradient.
// Thread = channel, block (x, y) = (channels, chunk of rows).
template <typename T>
__global__ __launch_bounds__(kBT) void k_norm_dw(BlockBwdParams p)
{
    const int64_t c = static_cast<int64_t>(blockIdx.x) * kBT + threadIdx.x;
    if (c >= p.C) return;
    const int64_t r0 = static_cast<int64_t>(blockIdx.y) * kRowsPerChunk;
    const int64_t r1 = r0 + kRowsPerChunk < p.rows ? r0 + kRowsPerChunk : p.rows;
    const int64_t gpr = p.C / p.group, grp = c / p.group;
    float acc = 0.f, zv, yv;
    for (int64_t r = r0; r < r1; ++r) {
        const int64_t i = r * p.C + c;
        acc += ldv<T>(p.dout, i) * gated<T>(p, i, &zv, &yv) * p.inv_rms[r * gpr + grp];
    }
    p.dw_part[blockIdx.y * p.C + c] = acc;
}

// out[c] = sum over k of part[k][c], k in order.
__global__ __launch_bounds__(kBT) void k_sum_chunks(const float* part, int64_t nchunks, int64_t ncols, float* out)
{
    const int64_t c = static_cast<int64_t>(blockIdx.x) * kBT + threadIdx.x;
    if (c >= ncols) return;
    float s = 0.f;
    for (int64_t k = 0; k < nchunks; ++k) s += part[k * ncols + c];
    out[c] = s;
}

unsigned blocks(int64_t n) { return static_cast<unsigned>((n + kBT - 1) / kBT); }

template <typename T>
hipError_t dt_apply(const BlockBwdParams& p, hipStream_t st)
{
    hipLaunchKernelGGL(k_dt_apply<T>, dim3(blocks(p.rows * p.H)), dim3(kBT), 0, st, p);
    return hipGetLastError();
}

template <typename T>
hipError_t out_side(const BlockBwdParams& p, hipStream_t st)
{
    if (p.group == 0) {
        hipLaunchKernelGGL(k_gate_bwd<T>, dim3(blocks(p.rows * p.C)), dim3(kBT), 0, st, p);
        return hipGetLastError();
    }
    int seg = 1, log2seg = 0;
    while (seg < p.group && seg < 64) {
        seg <<= 1;
        ++log2seg;
    }
    const int64_t per_block = (kBT / 64) * (64 / seg);
    const int64_t ngroups = p.rows * (p.C / p.group);
    hipLaunchKernelGGL(k_norm_bwd<T>, dim3(static_cast<unsigned>((ngroups + per_block - 1) / per_block)), dim3(kBT),
                       0, st, p, seg, log2seg);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !p.dw) return e;
    const int64_t nch = (p.rows + kRowsPerChunk - 1) / kRowsPerChunk;
    hipLaunchKernelGGL(k_norm_dw<T>, dim3(blocks(p.C), static_cast<unsigned>(nch)), dim3(kBT), 0, st, p);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_sum_chunks, dim3(blocks(p.C)), dim3(kBT), 0, st, p.dw_part, nch, p.C, p.dw);
    return hipGetLastError();
}

template <typename T>
hipError_t dt_side(const BlockBwdParams& p, hipStream_t st)
{
    const int64_t nch = (p.rows + kRowsPerChunk - 1) / kRowsPerChunk;
    hipLaunchKernelGGL(k_dt_bwd<T>, dim3(blocks(p.H), static_cast<unsigned>(nch)), dim3(kBT), 0, st, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !p.ddt_bias) return e;
    hipLaunchKernelGGL(k_sum_chunks, dim3(blocks(p.H)), dim3(kBT), 0, st, p.dbias_part, nch, p.H, p.ddt_bias);
    return hipGetLastError();
}

}  // namespace

int64_t block_bwd_row_chunks(int64_t rows) { return (rows + kRowsPerChunk - 1) / kRowsPerChunk; }

hipError_t launch_block_dt_apply(const BlockBwdParams& p, bool bf16, hipStream_t st)
{
    return bf16 ? dt_apply<uint16_t>(p, st) : dt_apply<float>(p, st);
}

hipError_t launch_block_out_bwd(const BlockBwdParams& p, bool bf16, hipStream_t st)
{
    return bf16 ? out_side<uint16_t>(p, st) : out_side<float>(p, st);
}

hipError_t launch_block_dt_bwd(const BlockBwdParams& p, bool bf16, hipStream_t st)
{
    return bf16 ? dt_side<uint16_t>(p, st) : dt_side<float>(p, st);
}

}  // namespace ssd
