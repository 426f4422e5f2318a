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
//
// What the block steps exchange with the layer -- dt after the dt step, the
// layer's output y, its gradient dy and the layer's ddt -- is float32 in every
// case (with bf16 activations too): only the block's own inputs and outputs
// (dt_raw, z, dout, dz, d dt_raw) have the activation dtype, so the result is
// the gradient of the block forward, which keeps dt and y in float32 as well.
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
    const float e = __expf(-fabsf(v));
    const float r = __builtin_amdgcn_rcpf(1.f + e);   // v_rcp_f32 (1 ulp)
    return v >= 0.f ? r : e * r;
}

// Eight consecutive channels (one 16- or 32-byte vector).
template <typename T>
__device__ __forceinline__ void load8(const void* p, int64_t i, float* v)
{
    if constexpr (sizeof(T) == 2) {
        const uint4 u = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(p) + i);
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            v[2 * k] = __uint_as_float(w[k] << 16);
            v[2 * k + 1] = __uint_as_float(w[k] & 0xFFFF0000u);
        }
    } else {
        const float4 a = *reinterpret_cast<const float4*>(static_cast<const float*>(p) + i);
        const float4 b = *reinterpret_cast<const float4*>(static_cast<const float*>(p) + i + 4);
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
        v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    }
}

template <typename T>
__device__ __forceinline__ void store8(void* p, int64_t i, const float* v)
{
    if constexpr (sizeof(T) == 2) {
        uint32_t w[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            uint32_t lo = __float_as_uint(v[2 * k]), hi = __float_as_uint(v[2 * k + 1]);
            lo = (lo + 0x7FFFu + ((lo >> 16) & 1u)) >> 16;   // nearest even
            hi = (hi + 0x7FFFu + ((hi >> 16) & 1u)) >> 16;
            w[k] = lo | (hi << 16);
        }
        *reinterpret_cast<uint4*>(static_cast<uint16_t*>(p) + i) = make_uint4(w[0], w[1], w[2], w[3]);
    } else {
        *reinterpret_cast<float4*>(static_cast<float*>(p) + i) = make_float4(v[0], v[1], v[2], v[3]);
        *reinterpret_cast<float4*>(static_cast<float*>(p) + i + 4) = make_float4(v[4], v[5], v[6], v[7]);
    }
}

template <int CTRL>
__device__ __forceinline__ float dpp_add(float v)
{
    return v + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

__device__ __forceinline__ float swap_add(float v, bool rows16)
{
    const uint32_t u = __float_as_uint(v);
    const auto a = rows16 ? __builtin_amdgcn_permlane16_swap(u, u, false, false)
                          : __builtin_amdgcn_permlane32_swap(u, u, false, false);
    return __uint_as_float(a[0]) + __uint_as_float(a[1]);
}

// Sum over aligned segments of `seg` lanes (a power of two, at most 64), in
// registers; every lane of a segment gets the segment's sum.  The same fixed
// sequence of steps for every segment (deterministic).
__device__ __forceinline__ float segment_sum(float v, int seg)
{
    if (seg >= 2) v = dpp_add<0xB1>(v);    // quad_perm [1,0,3,2]: lane ^ 1
    if (seg >= 4) v = dpp_add<0x4E>(v);    // quad_perm [2,3,0,1]: lane ^ 2
    if (seg >= 8) v = dpp_add<0x141>(v);   // row_half_mirror: the other quad of the 8
    if (seg >= 16) v = dpp_add<0x140>(v);  // row_mirror: the other half of the row
    if (seg >= 32) v = swap_add(v, true);  // the neighbouring row
    if (seg >= 64) v = swap_add(v, false); // the other half of the wavefront
    return v;
}

// The dt step of the forward, into a float32 buffer.
template <typename T>
__global__ __launch_bounds__(kBT) void k_dt_apply(BlockBwdParams p)
{
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kBT + threadIdx.x;
    if (i >= p.rows * p.H) return;
    const int64_t h = i % p.H;
    float v = ldv<T>(p.dt_raw, i) + (p.bias ? p.bias[h] : 0.f);
    if (p.softplus) v = softplus_f(v);
    static_cast<float*>(p.dt)[i] = fminf(fmaxf(v, p.lo), p.hi);
}

// bf16 -> float32 (exact) and float32 -> bf16 (nearest even), one element
// per thread (any length and alignment).
__global__ __launch_bounds__(kBT) void k_widen(const void* src, float* dst, int64_t n)
{
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kBT + threadIdx.x;
    if (i < n) dst[i] = ldv<uint16_t>(src, i);
}

__global__ __launch_bounds__(kBT) void k_narrow(const float* src, void* dst, int64_t n)
{
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kBT + threadIdx.x;
    if (i < n) stv<uint16_t>(dst, i, src[i]);
}

// d dt_raw, and per-chunk partial sums over rows for d bias.  Thread = head,
// block (x, y) = (heads, chunk of kRowsPerChunk rows).
constexpr int kRowsPerChunk = 16;

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
        const float dv = in ? static_cast<const float*>(p.ddt)[i] * (p.softplus ? sigmoid_f(v) : 1.f) : 0.f;
        stv<T>(p.ddt_raw, i, dv);
        acc += dv;
    }
    if (p.dbias_part) p.dbias_part[blockIdx.y * p.H + h] = acc;
}

// Gate only: dy = dout SiLU(z), dz = dout y SiLU'(z), eight channels per thread.
template <typename T>
__global__ __launch_bounds__(kBT) void k_gate_bwd(BlockBwdParams p)
{
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kBT + threadIdx.x;
    if (i >= p.rows * p.C / 8) return;
    float y[8], z[8], d[8], dy[8], dz[8];
    load8<float>(p.y, 8 * i, y);
    load8<T>(p.z, 8 * i, z);
    load8<T>(p.dout, 8 * i, d);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const float s = sigmoid_f(z[e]);
        dy[e] = d[e] * z[e] * s;
        dz[e] = d[e] * y[e] * s * (1.f + z[e] * (1.f - s));
    }
    store8<float>(p.dy, 8 * i, dy);
    store8<T>(p.dz, 8 * i, dz);
}

// One piece (8 channels) of a group: y, z and sigmoid(z) (when gating), the
// gated value, dout.
template <typename T>
struct Piece {
    float y[8], z[8], s[8], gv[8], d[8];
    __device__ __forceinline__ void load(const BlockBwdParams& p, int64_t e)
    {
        load8<float>(p.y, e, y);
        load8<T>(p.dout, e, d);
        if (p.z) {
            load8<T>(p.z, e, z);
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                s[k] = sigmoid_f(z[k]);
                gv[k] = y[k] * z[k] * s[k];
            }
        } else {
#pragma unroll
            for (int k = 0; k < 8; ++k) gv[k] = y[k];
        }
    }
    __device__ __forceinline__ float g(const BlockBwdParams&, int k) const { return gv[k]; }
};

// Normalisation (after the optional gate): a group of `group` channels is
// group / 8 pieces spread over `seg` lanes (a power of two, at most 64); each
// lane keeps its (at most MAXP) pieces in registers through the three steps
// (sum of squares; sum of dn n; the gradients), or re-reads them when the
// group is wider (MAXP == 0).  Records 1 / r per (row, group) for the weight
// gradient.
// The gradients of one (row, group), by the `seg` lanes that hold it.  acc
// (may be null): this lane's pieces' dout n added to it, for the weight
// gradient.  Every lane of the wavefront takes part (cross-lane sums); lanes of
// an inactive group load and store nothing.
template <typename T, int MAXP>
__device__ __forceinline__ void norm_group_bwd(const BlockBwdParams& p, bool active, int64_t gid, int64_t row,
                                               int64_t c0, int li, int seg, float* acc)
{
    const int64_t base = row * p.C + c0;
    const int pieces = static_cast<int>(p.group / 8);
    Piece<T> pc[MAXP > 0 ? MAXP : 1];
    const int mine = active ? (pieces - li + seg - 1) / seg : 0;   // pieces of this lane
    // f(piece, j) over this lane's pieces j = li, li + seg, ...: from registers,
    // or re-read when the group is too wide to keep them
    const auto each_piece = [&](auto&& f) {
        if constexpr (MAXP > 0) {
#pragma unroll
            for (int k = 0; k < MAXP; ++k)
                if (k < mine) f(pc[k], li + k * seg);
        } else {
            for (int k = 0; k < mine; ++k) {
                pc[0].load(p, base + 8 * (li + k * seg));
                f(pc[0], li + k * seg);
            }
        }
    };
    const auto weights = [&](int j, float* w) {
        if (p.w) {
            const float4 w0 = *reinterpret_cast<const float4*>(p.w + c0 + 8 * j);
            const float4 w1 = *reinterpret_cast<const float4*>(p.w + c0 + 8 * j + 4);
            w[0] = w0.x; w[1] = w0.y; w[2] = w0.z; w[3] = w0.w;
            w[4] = w1.x; w[5] = w1.y; w[6] = w1.z; w[7] = w1.w;
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) w[e] = 1.f;
        }
    };
    if constexpr (MAXP > 0) {
#pragma unroll
        for (int k = 0; k < MAXP; ++k)
            if (k < mine) pc[k].load(p, base + 8 * (li + k * seg));
    }
    float ss = 0.f;
    each_piece([&](const Piece<T>& q, int) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float g = q.g(p, e);
            ss += g * g;
        }
    });
    ss = segment_sum(ss, seg);
    const float inv = 1.f / sqrtf(ss / static_cast<float>(p.group) + p.eps);
    float sdn = 0.f;
    each_piece([&](const Piece<T>& q, int j) {
        float w[8];
        weights(j, w);
#pragma unroll
        for (int e = 0; e < 8; ++e) sdn += q.d[e] * w[e] * q.g(p, e) * inv;
    });
    sdn = segment_sum(sdn, seg);
    if (!active) return;
    const float mdn = sdn / static_cast<float>(p.group);
    each_piece([&](const Piece<T>& q, int j) {
        float w[8], dy[8], dz[8];
        weights(j, w);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float n = q.g(p, e) * inv;
            const float dg = (q.d[e] * w[e] - n * mdn) * inv;
            if (p.z) {
                const float s = q.s[e];
                dy[e] = dg * q.z[e] * s;
                dz[e] = dg * q.y[e] * s * (1.f + q.z[e] * (1.f - s));
            } else {
                dy[e] = dg;
            }
        }
        store8<float>(p.dy, base + 8 * j, dy);
        if (p.z) store8<T>(p.dz, base + 8 * j, dz);
    });
    if (li == 0 && p.inv_rms) p.inv_rms[gid] = inv;
    if constexpr (MAXP > 0) {
        if (acc) {
#pragma unroll
            for (int k = 0; k < MAXP; ++k)
                if (k < mine)
#pragma unroll
                    for (int e = 0; e < 8; ++e) acc[8 * k + e] += pc[k].d[e] * pc[k].g(p, e) * inv;
        }
    }
}

template <typename T, int MAXP>
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
    norm_group_bwd<T, MAXP>(p, active, gid, row, c0, li, seg, nullptr);
}

// The same with the weight gradient's per-chunk partial sums folded in (groups
// of at most 2 pieces per lane): workgroup (x, y) = (a run of groups of a row,
// chunk of kRowsPerChunk rows); each segment keeps its group over the chunk's
// rows and adds dout n in registers, so y, z and dout are read once.
template <typename T, int MAXP>
__global__ __launch_bounds__(kBT) void k_norm_bwd_rows(BlockBwdParams p, int seg, int log2seg)
{
    static_assert(MAXP > 0, "pieces kept in registers");
    const int lane = threadIdx.x & 63;
    const int per_wave = 64 >> log2seg;
    const int64_t gpr = p.C / p.group;
    const int64_t g = (static_cast<int64_t>(blockIdx.x) * (kBT / 64) + (threadIdx.x >> 6)) * per_wave +
                      (lane >> log2seg);
    const int li = lane & (seg - 1);
    const bool active = g < gpr;
    const int64_t c0 = active ? g * p.group : 0;
    const int64_t r0 = static_cast<int64_t>(blockIdx.y) * kRowsPerChunk;
    const int64_t r1 = r0 + kRowsPerChunk < p.rows ? r0 + kRowsPerChunk : p.rows;
    float acc[8 * MAXP];
#pragma unroll
    for (int k = 0; k < 8 * MAXP; ++k) acc[k] = 0.f;
    for (int64_t r = r0; r < r1; ++r) norm_group_bwd<T, MAXP>(p, active, r * gpr + g, r, c0, li, seg, acc);
    if (!active) return;
    const int pieces = static_cast<int>(p.group / 8);
    const int mine = (pieces - li + seg - 1) / seg;
    float* o = p.dw_part + static_cast<int64_t>(blockIdx.y) * p.C + c0;
#pragma unroll
    for (int k = 0; k < MAXP; ++k)
        if (k < mine) {
            const int j = li + k * seg;
            *reinterpret_cast<float4*>(o + 8 * j) = make_float4(acc[8 * k], acc[8 * k + 1], acc[8 * k + 2], acc[8 * k + 3]);
            *reinterpret_cast<float4*>(o + 8 * j + 4) =
                make_float4(acc[8 * k + 4], acc[8 * k + 5], acc[8 * k + 6], acc[8 * k + 7]);
        }
}

// Per-chunk partial sums over rows of dout n for the weight gradient.  Thread =
// 8 channels, block (x, y) = (channels, chunk of kRowsPerChunk rows).
template <typename T>
__global__ __launch_bounds__(kBT) void k_norm_dw(BlockBwdParams p)
{
    const int64_t c8 = static_cast<int64_t>(blockIdx.x) * kBT + threadIdx.x;
    if (c8 >= p.C / 8) return;
    const int64_t r0 = static_cast<int64_t>(blockIdx.y) * kRowsPerChunk;
    const int64_t r1 = r0 + kRowsPerChunk < p.rows ? r0 + kRowsPerChunk : p.rows;
    const int64_t gpr = p.C / p.group, grp = 8 * c8 / p.group;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int64_t r = r0; r < r1; ++r) {
        Piece<T> q;
        q.load(p, r * p.C + 8 * c8);
        const float inv = p.inv_rms[r * gpr + grp];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += q.d[e] * q.g(p, e) * inv;
    }
    float* o = p.dw_part + blockIdx.y * p.C + 8 * c8;
    *reinterpret_cast<float4*>(o) = make_float4(acc[0], acc[1], acc[2], acc[3]);
    *reinterpret_cast<float4*>(o + 4) = make_float4(acc[4], acc[5], acc[6], acc[7]);
}

// out[c] = sum over k of part[k][c]: one block per column, thread t takes
// k = t, t + 256, ... in order, then a fixed tree over the block.
__global__ __launch_bounds__(kBT) void k_sum_chunks(const float* part, int64_t nchunks, int64_t ncols, float* out)
{
    __shared__ float scr[kBT / 64];
    const int64_t c = blockIdx.x;
    float s = 0.f;
    for (int64_t k = threadIdx.x; k < nchunks; k += kBT) s += part[k * ncols + c];
    s = segment_sum(s, 64);
    if ((threadIdx.x & 63) == 0) scr[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) out[c] = (scr[0] + scr[1]) + (scr[2] + scr[3]);
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
        hipLaunchKernelGGL(k_gate_bwd<T>, dim3(blocks(p.rows * p.C / 8)), dim3(kBT), 0, st, p);
        return hipGetLastError();
    }
    const int64_t pieces = p.group / 8;
    int seg = 1, log2seg = 0;
    while (seg < pieces && seg < 64) {
        seg <<= 1;
        ++log2seg;
    }
    const int64_t per_block = (kBT / 64) * (64 / seg);
    const int64_t ngroups = p.rows * (p.C / p.group);
    const dim3 grid(static_cast<unsigned>((ngroups + per_block - 1) / per_block));
    const int64_t per_lane = (pieces + seg - 1) / seg;
    const int64_t nch = (p.rows + kRowsPerChunk - 1) / kRowsPerChunk;
    if (p.dw && per_lane <= 2) {   // weight gradient folded in: y, z, dout read once
        const int64_t gpr = p.C / p.group;
        const dim3 g2(static_cast<unsigned>((gpr + per_block - 1) / per_block), static_cast<unsigned>(nch));
        if (per_lane <= 1)
            hipLaunchKernelGGL((k_norm_bwd_rows<T, 1>), g2, dim3(kBT), 0, st, p, seg, log2seg);
        else
            hipLaunchKernelGGL((k_norm_bwd_rows<T, 2>), g2, dim3(kBT), 0, st, p, seg, log2seg);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(k_sum_chunks, dim3(static_cast<unsigned>(p.C)), dim3(kBT), 0, st, p.dw_part, nch, p.C,
                           p.dw);
        return hipGetLastError();
    }
    if (per_lane <= 1)
        hipLaunchKernelGGL((k_norm_bwd<T, 1>), grid, dim3(kBT), 0, st, p, seg, log2seg);
    else if (per_lane <= 2)
        hipLaunchKernelGGL((k_norm_bwd<T, 2>), grid, dim3(kBT), 0, st, p, seg, log2seg);
    else
        hipLaunchKernelGGL((k_norm_bwd<T, 0>), grid, dim3(kBT), 0, st, p, seg, log2seg);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !p.dw) return e;
    hipLaunchKernelGGL(k_norm_dw<T>, dim3(blocks(p.C / 8), static_cast<unsigned>(nch)), dim3(kBT), 0, st, p);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_sum_chunks, dim3(static_cast<unsigned>(p.C)), dim3(kBT), 0, st, p.dw_part, nch, p.C, p.dw);
    return hipGetLastError();
}

template <typename T>
hipError_t dt_side(const BlockBwdParams& p, hipStream_t st)
{
    const int64_t nch = (p.rows + kRowsPerChunk - 1) / kRowsPerChunk;
    hipLaunchKernelGGL(k_dt_bwd<T>, dim3(blocks(p.H), static_cast<unsigned>(nch)), dim3(kBT), 0, st, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !p.ddt_bias) return e;
    hipLaunchKernelGGL(k_sum_chunks, dim3(static_cast<unsigned>(p.H)), dim3(kBT), 0, st, p.dbias_part, nch, p.H,
                       p.ddt_bias);
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

hipError_t launch_widen(const void* src, float* dst, int64_t n, hipStream_t st)
{
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_widen, dim3(blocks(n)), dim3(kBT), 0, st, src, dst, n);
    return hipGetLastError();
}

hipError_t launch_narrow(const float* src, void* dst, int64_t n, hipStream_t st)
{
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_narrow, dim3(blocks(n)), dim3(kBT), 0, st, src, dst, n);
    return hipGetLastError();
}

}  // namespace ssd
