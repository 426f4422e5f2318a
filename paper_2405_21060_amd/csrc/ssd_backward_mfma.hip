// Gradients of the SSD layer on the matrix cores: bf16 inputs, headdim 64,
// dstate 64 or 128.  Same chunked adjoint as ssd_backward.hip (formulas at the
// top of that file), with chunks of 64 tokens and every contraction on
// v_mfma_f32_16x16x32_bf16 (bf16 operands, float32 accumulation):
//
//   k_bwd2_pass    the chunk states: per (row, head, direction) a walk
//                  over the chunks with a float32 running
//                  state, writing h_in^T (forward) or Gn^T (backward, from the
//                  final-state gradient) per chunk in bf16; the initial-state
//                  gradient in float32
//   k_bwd2_chunk   per (chunk, row, group, head slice): all chunk terms.  Score
//                  tiles (u >= t) R0 = dy x^T and G0 = C B^T (once per
//                  workgroup), then dX~^T = dy^T Gs + Gn B^T, dB^T = C^T Rs +
//                  Gn^T x~^T, dC^T = B^T Rs^T + h_in^T dy^T, each as 16 x 16
//                  tiles whose operands are k-contiguous rows: in shared memory
//                  (B, B^T, C^T, x, dy, dy^T, the score tiles and Gn, transposed
//                  there from Gn^T), or straight from global memory (Gn^T, h_in^T).
//
// H32 (a template flag; the block gradients use it): dt and dy come in as
// float32 and ddt goes out as float32.  dy is rounded to bf16 only where it is
// a matrix-core operand; the skip term of dx and the dD sums take it in float32.
//
// An MFMA operand row holds the contraction index contiguously; a lane
// (row r = lane % 16, group q = lane / 16) reads 8 of them (k = 32 s + 8 q ..
// + 7) as one 16-byte load, and the result tile D[4 q + v][r] lands in its
// four accumulator registers.  Shared arrays are padded by 8 elements per
// row so that the 16 rows of a fragment read fall in distinct banks.
#include <type_traits>

#include "ssd_bwd.h"
#include "ssd_device.h"

namespace ssd {
namespace {

constexpr int kQ2 = 64;          // tokens per chunk
constexpr int kP2 = 64;          // head dimension
constexpr int kT2 = 512;         // threads per workgroup (8 wavefronts)
constexpr int kLd = kQ2 + 8;     // row stride (elements) of 64-wide shared rows

typedef uint16_t u16;

__device__ __forceinline__ bf16x8_t frag(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }

__device__ __forceinline__ f32x4_t mma(uint4 a, uint4 b, f32x4_t c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(frag(a), frag(b), c, 0, 0, 0);
}

__device__ __forceinline__ uint32_t bf16_bits(float f)
{
    uint32_t u = __float_as_uint(f);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;   // nearest even (finite inputs)
}

__device__ __forceinline__ uint32_t pack2(float lo, float hi) { return bf16_bits(lo) | (bf16_bits(hi) << 16); }

__device__ __forceinline__ float bf(u16 v) { return __uint_as_float(static_cast<uint32_t>(v) << 16); }

// Two floats rounded to bf16 (nearest even; the inputs are finite), the first
// in the low half.
__device__ __forceinline__ uint32_t rne_pair(float a, float b)
{
    uint32_t ua = __float_as_uint(a), ub = __float_as_uint(b);
    ua += 0x7FFFu + ((ua >> 16) & 1u);
    ub += 0x7FFFu + ((ub >> 16) & 1u);
    return (ua >> 16) | (ub & 0xFFFF0000u);
}

// dt of token row i (bf16 bits, or float32 with H32).
template <bool H32>
__device__ __forceinline__ float load_dt(const void* dt, int64_t i)
{
    if constexpr (H32)
        return static_cast<const float*>(dt)[i];
    else
        return bf(static_cast<const u16*>(dt)[i]);
}

// dt as raw bits (float32, or bf16 in the low half), widened where it is used:
// a load whose value is converted at once makes the wavefront wait for every
// memory operation issued before it (the prefetches and the state stores).
template <bool H32>
__device__ __forceinline__ uint32_t load_dt_raw(const void* dt, int64_t i)
{
    if constexpr (H32)
        return __float_as_uint(static_cast<const float*>(dt)[i]);
    else
        return static_cast<const u16*>(dt)[i];
}

template <bool H32>
__device__ __forceinline__ float dt_of_raw(uint32_t v)
{
    return H32 ? __uint_as_float(v) : __uint_as_float(v << 16);
}

__device__ __forceinline__ float lo_f(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_f(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// One operand fragment of a row-major bf16 array: row `row`, k-step `ks`.
__device__ __forceinline__ uint4 ldfrag(const u16* a, int ld, int row, int ks, int lane)
{
    return *reinterpret_cast<const uint4*>(a + row * ld + ks * 32 + 8 * (lane >> 4));
}

__device__ __forceinline__ uint4 ldfrag_g(const u16* a, int64_t ld, int row, int ks, int lane)
{
    return *reinterpret_cast<const uint4*>(a + static_cast<int64_t>(row) * ld + ks * 32 + 8 * (lane >> 4));
}

// Cross-lane sums in registers (DPP and the permlane swaps; no trip through
// shared memory).
template <int CTRL, int ROWS>
__device__ __forceinline__ float dpp(float v)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, ROWS, 0xF, false));
}

// Sum over the 16 lanes of each row (row_ror by 8, 4, 2, 1): every lane of the row gets it.
__device__ __forceinline__ float row_sum16(float v)
{
    v += dpp<0x128, 0xF>(v);
    v += dpp<0x124, 0xF>(v);
    v += dpp<0x122, 0xF>(v);
    v += dpp<0x121, 0xF>(v);
    return v;
}

// Sum over the four rows at each position (lanes r, r + 16, r + 32, r + 48):
// swapping odd rows with even ones, then the halves, and adding.
__device__ __forceinline__ float col_sum4(float v)
{
    uint32_t u = __float_as_uint(v);
    const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    u = __float_as_uint(v);
    const auto b = __builtin_amdgcn_permlane32_swap(u, u, false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Sum over the 64 lanes of a wavefront (every lane gets it).
__device__ __forceinline__ float wave_sum(float v) { return col_sum4(row_sum16(v)); }

// Inclusive prefix sum over the 64 lanes: shifts by 1, 2, 4, 8 within each
// row, then the row totals carried up by broadcasts of lanes 15 (into rows 1
// and 3) and 31 (into rows 2 and 3).  Lanes with no source add zero.
__device__ __forceinline__ float wave_scan(float v)
{
    v += dpp<0x111, 0xF>(v);
    v += dpp<0x112, 0xF>(v);
    v += dpp<0x114, 0xF>(v);
    v += dpp<0x118, 0xF>(v);
    v += dpp<0x142, 0xA>(v);
    v += dpp<0x143, 0xC>(v);
    return v;
}

__device__ __forceinline__ float lane_value(float v, int lane)
{
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

__device__ __forceinline__ int chunk_len2(int64_t T, int64_t c)
{
    const int64_t r = T - c * kQ2;
    return static_cast<int>(r < kQ2 ? r : kQ2);
}

// Slice of a group's heads handled by this workgroup.
struct HeadRange {
    int64_t g, slice, lo, hi;
};

__device__ __forceinline__ HeadRange head_range(const BwdParams& p)
{
    HeadRange r;
    const int64_t hpg = p.H / p.G;
    r.g = blockIdx.z / p.S;
    r.slice = blockIdx.z - r.g * p.S;
    r.lo = r.g * hpg + r.slice * p.hs;
    r.hi = (r.slice + 1) * p.hs < hpg ? r.lo + p.hs : r.g * hpg + hpg;
    return r;
}

// ---------------------------------------------------------------------------
// State passes: one workgroup per (row, head, direction) walks the chunks in
// order with a float32 running state S (64 p x N) in registers, and writes S
// (bf16, n x p) for every chunk before adding the chunk's own term:
//   direction 0 (forward, from the initial state): h_in(c) = S, then
//     S <- exp(cs_end) S + sum_s (e(end,s) dt_s x_s) B_s^T;
//   direction 1 (backward, from the final-state gradient): Gn(c) = S, then
//     S <- exp(cs_end) S + sum_u (exp(cs_u) dy_u) C_u^T;
//   at the end of direction 1, S is the initial-state gradient (float32).
// The chunk term is a 64 x N x 64 product over the chunk's tokens on the
// matrix cores.  Both operands stay token-major in shared memory (whole
// 16-byte pieces of rows, as loaded: the global loads are coalesced), with
// each row's 8-element groups XOR-swizzled by the row index, and the
// contraction fragments come out of transposing reads (ds_read_b64_tr_b16):
// within a 16-lane group, source lane j reads row k0 + j/4, elements f0 +
// 4 (j%4) .. +3, and lane i receives element f0 + i of rows k0 .. k0 + 3.
// Lane group g takes rows 4 g .. 4 g + 3 and 16 + 4 g .. 16 + 4 g + 3 of each
// 32-token step for its eight contraction slots (the same map for both
// operands).  Inputs are fetched two chunks ahead.  Wavefront w owns p rows
// 16 w .. 16 w + 15 of S (N / 16 tiles of 16 x 16).
constexpr int kPassT = 256;

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

// Element offset of (row s, element f) in a token-major buffer of F elements
// per row, 8-element groups swizzled by (s & 7).
template <int F>
__device__ __forceinline__ int tok_off(int s, int f)
{
    return s * F + ((((f >> 3) ^ (s & 7)) << 3) | (f & 7));
}

// Contraction fragment over tokens 32 m .. 32 m + 31 of elements f0 .. f0 + 15.
template <int F>
__device__ __forceinline__ uint4 tr_frag(const u16* buf, int m, int f0, int lane)
{
    const int j = lane & 15, g = lane >> 4;
    const int row = 32 * m + 4 * g + (j >> 2), f = f0 + 4 * (j & 3);
    const uint2 lo = __builtin_bit_cast(
        uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(buf + tok_off<F>(row, f))));
    const uint2 hi = __builtin_bit_cast(
        uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(buf + tok_off<F>(row + 16, f))));
    return make_uint4(lo.x, lo.y, hi.x, hi.y);
}

// PACKED: a packed row; workgroup (sequence, head) walks that sequence's
// chunks of the chunk table.
template <int N, bool PACKED, bool H32>
__global__ __launch_bounds__(kPassT, H32 ? 2 : 1) void k_bwd2_pass(BwdParams p)
{
    __shared__ __attribute__((aligned(16))) u16 XS[kQ2 * kP2];   // weighted x (or dy), token-major
    __shared__ __attribute__((aligned(16))) u16 YS[kQ2 * N];     // B (or C), token-major
    // the chunk's state (bf16, n x p) on its way out: rows padded to 72
    // elements so that the 16 n-rows of a wavefront's writes spread over the
    // banks; read back as whole 128-byte rows, so that the global stores cover
    // full rows (a wavefront's own fragments are 32-byte pieces of 16 rows)
    constexpr int kOBld = kP2 + 8;
    __shared__ __attribute__((aligned(16))) u16 OB[N * kOBld];

    const int64_t bh = blockIdx.x;
    const int64_t b = bh / p.H, h = bh - b * p.H, g = h / (p.H / p.G);
    const int dir = static_cast<int>(blockIdx.y);
    // wavefront index, provably uniform (per-wavefront choices stay scalar)
    const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane & 15, q = lane >> 4;
    const u16* src = static_cast<const u16*>(dir == 0 ? p.x : p.dy);
    const float* dyf = static_cast<const float*>(p.dy);   // H32, dir 1
    const bool src32 = H32 && dir == 1;
    const u16* bc = static_cast<const u16*>(dir == 0 ? p.B : p.C);
    u16* out = reinterpret_cast<u16*>(dir == 0 ? p.hin : p.gnT);
    const float A2 = -expf(p.A_log[h]) * kLog2e;

    // running state: lane holds S[p = 16 w + 4 q + v][n = 16 nt + r]
    constexpr int kNT = N / 16;
    f32x4_t S[kNT];
    const float* s0 = dir == 0 ? p.init : p.dfinal;
#pragma unroll
    for (int nt = 0; nt < kNT; ++nt)
#pragma unroll
        for (int v = 0; v < 4; ++v)
            S[nt][v] = s0 ? s0[(bh * kP2 + 16 * w + 4 * q + v) * N + 16 * nt + r] : 0.f;

    // The passes' loop, once per kind of source (the float32 dy of the block
    // gradients' direction 1 is known per workgroup): no branch on it inside
    // the loop, whose waits then count the loads in flight.
    const auto run = [&](auto s32tag) {
        constexpr bool S32 = decltype(s32tag)::value;
        // One chunk's inputs: dt (lane = token), and 16-byte pieces of x (or dy)
        // and of B (or C): piece i = tid + 256 k is row i / (F/8), group i % (F/8),
        // so consecutive lanes read consecutive bytes of a row.
        constexpr int kXK = kQ2 * kP2 / 8 / kPassT;   // 2
        constexpr int kYK = kQ2 * N / 8 / kPassT;     // N / 32
        struct Stage {
            uint32_t dt;   // raw bits (see load_dt_raw)
            uint4 x[kXK], y[kYK];
            float4 xf[H32 ? 2 * kXK : 1];   // H32, dir 1: dy in float32
        };
        int64_t first = 0, nch = p.nC;   // this row's (or sequence's) chunks
        if constexpr (PACKED) {
            first = p.seq_first[b];
            nch = p.seq_first[b + 1] - first;
        }
        const auto chunk_at = [&](int64_t k) { return first + (dir == 0 ? k : nch - 1 - k); };
        const auto fetch = [&](Stage& st, int64_t k) {
            // Branch-free: past the last chunk the last one is fetched again (never
            // used), and rows past a partial chunk read as zeros through the buffer
            // bounds, so that the compiler can count exactly which loads are still
            // in flight when a stage is used (with branches around them it waits
            // for all of them: the next stage's and the state stores included).
            const int64_t c = chunk_at(k < nch ? k : nch - 1);
            int L;
            int64_t t0;
            if constexpr (PACKED) {
                const int4 e = p.vtab[c];
                L = e.y;
                t0 = e.x;
            } else {
                L = chunk_len2(p.T, c);
                t0 = b * p.T + c * kQ2;
            }
            constexpr int kDtBytes = H32 ? 4 : 2;
            const __amdgpu_buffer_rsrc_t rdt = __builtin_amdgcn_make_buffer_rsrc(
                const_cast<char*>(static_cast<const char*>(p.dt)) + (t0 * p.H + h) * kDtBytes, 0,
                static_cast<int>(((L - 1) * p.H + 1) * kDtBytes), 0x00020000);
            const int dtoff = lane * static_cast<int>(p.H) * kDtBytes;
            if constexpr (H32)
                st.dt = __builtin_amdgcn_raw_buffer_load_b32(rdt, dtoff, 0, 0);
            else
                st.dt = __builtin_amdgcn_raw_buffer_load_b16(rdt, dtoff, 0, 0);
            const int xrow = static_cast<int>(p.H) * kP2;   // elements between tokens of x (dy)
    #pragma unroll
            for (int kk = 0; kk < kXK; ++kk) {
                const int i = tid + kPassT * kk, s = i >> 3, f = 8 * (i & 7);
                if constexpr (S32) {
                    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
                        const_cast<float*>(dyf) + (t0 * p.H + h) * kP2, 0,
                        ((L - 1) * xrow + kP2) * static_cast<int>(sizeof(float)), 0x00020000);
                    const int off = (s * xrow + f) * static_cast<int>(sizeof(float));
                    st.xf[2 * kk] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
                    st.xf[2 * kk + 1] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rs, off + 16, 0, 0));
                } else {
                    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
                        const_cast<u16*>(src) + (t0 * p.H + h) * kP2, 0,
                        ((L - 1) * xrow + kP2) * static_cast<int>(sizeof(u16)), 0x00020000);
                    st.x[kk] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                                             rs, (s * xrow + f) * static_cast<int>(sizeof(u16)), 0, 0));
                }
            }
            const int yrow = static_cast<int>(p.G) * N;   // elements between tokens of B (C)
            const __amdgpu_buffer_rsrc_t ry = __builtin_amdgcn_make_buffer_rsrc(
                const_cast<u16*>(bc) + (t0 * p.G + g) * N, 0, ((L - 1) * yrow + N) * static_cast<int>(sizeof(u16)),
                0x00020000);
    #pragma unroll
            for (int kk = 0; kk < kYK; ++kk) {
                const int i = tid + kPassT * kk, s = i / (N / 8), f = 8 * (i % (N / 8));
                st.y[kk] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                                         ry, (s * yrow + f) * static_cast<int>(sizeof(u16)), 0, 0));
            }
        };
        const auto step = [&](Stage& st, int64_t k) {
            const int64_t c = chunk_at(k);
            const int L = PACKED ? p.vtab[c].y : chunk_len2(p.T, c);
            // token weights: cumsum with lane = token, then each piece's token's weight
            const float dtv = dt_of_raw<H32>(st.dt);
            const float cs = wave_scan(dtv * A2);
            const float csend = lane_value(cs, L - 1);
            const float wt = dir == 0 ? exp2f(csend - cs) * dtv : exp2f(cs);
            __syncthreads();   // the previous chunk's product is done with XS, YS
    #pragma unroll
            for (int kk = 0; kk < kXK; ++kk) {
                const int i = tid + kPassT * kk, s = i >> 3, f = 8 * (i & 7);
                const float ws = __shfl(wt, s, 64);
                uint32_t o[4];
                if constexpr (S32) {
                    const float4 a = st.xf[2 * kk], c2 = st.xf[2 * kk + 1];
                    o[0] = pack2(ws * a.x, ws * a.y);
                    o[1] = pack2(ws * a.z, ws * a.w);
                    o[2] = pack2(ws * c2.x, ws * c2.y);
                    o[3] = pack2(ws * c2.z, ws * c2.w);
                } else {
                    const uint32_t ex[4] = {st.x[kk].x, st.x[kk].y, st.x[kk].z, st.x[kk].w};
    #pragma unroll
                    for (int e = 0; e < 4; ++e) o[e] = pack2(ws * lo_f(ex[e]), ws * hi_f(ex[e]));
                }
                *reinterpret_cast<uint4*>(XS + tok_off<kP2>(s, f)) = make_uint4(o[0], o[1], o[2], o[3]);
            }
    #pragma unroll
            for (int kk = 0; kk < kYK; ++kk) {
                const int i = tid + kPassT * kk, s = i / (N / 8), f = 8 * (i % (N / 8));
                *reinterpret_cast<uint4*>(YS + tok_off<N>(s, f)) = st.y[kk];
            }
            fetch(st, k + 2);

            // S before this chunk's term -> out(c), bf16 (n x p), through OB
    #pragma unroll
            for (int nt = 0; nt < kNT; ++nt)
                *reinterpret_cast<uint2*>(OB + (16 * nt + r) * kOBld + 16 * w + 4 * q) =
                    make_uint2(pack2(S[nt][0], S[nt][1]), pack2(S[nt][2], S[nt][3]));

            __syncthreads();   // this chunk's operands and its state in place
            {
                u16* o = out + ((PACKED ? c : b * p.nC + c) * p.H + h) * kP2 * N;
                constexpr int kOK = N * kP2 / 8 / kPassT;   // 16-byte pieces per thread
    #pragma unroll
                for (int kk = 0; kk < kOK; ++kk) {
                    const int i = tid + kPassT * kk, row = i >> 3, c8 = 8 * (i & 7);
                    *reinterpret_cast<uint4*>(o + row * kP2 + c8) =
                        *reinterpret_cast<const uint4*>(OB + row * kOBld + c8);
                }
            }
            const float a = exp2f(csend);
            const uint4 xf0 = tr_frag<kP2>(XS, 0, 16 * w, lane), xf1 = tr_frag<kP2>(XS, 1, 16 * w, lane);
    #pragma unroll
            for (int nt = 0; nt < kNT; ++nt) {
                f32x4_t t = zero4();
                t = mma(xf0, tr_frag<N>(YS, 0, 16 * nt, lane), t);
                t = mma(xf1, tr_frag<N>(YS, 1, 16 * nt, lane), t);
    #pragma unroll
                for (int v = 0; v < 4; ++v) S[nt][v] = fmaf(a, S[nt][v], t[v]);
            }
        };
        Stage s0st, s1st;
        fetch(s0st, 0);
        fetch(s1st, 1);
        // (pairs of steps, then an odd last one: no branch inside the loop body)
        int64_t k = 0;
        for (; k + 1 < nch; k += 2) {
            step(s0st, k);
            step(s1st, k + 1);
        }
        if (k < nch) step(s0st, k);
    };
    if (src32)
        run(std::true_type{});
    else
        run(std::false_type{});
    if (dir == 1 && p.dinit) {
#pragma unroll
        for (int nt = 0; nt < kNT; ++nt)
#pragma unroll
            for (int v = 0; v < 4; ++v) p.dinit[(bh * kP2 + 16 * w + 4 * q + v) * N + 16 * nt + r] = S[nt][v];
    }
}

// ---------------------------------------------------------------------------
// Chunk gradients.
template <int N, bool H32 = false>
struct ChunkSmem {
    // Row strides (elements) of the shared tiles: N-wide rows (B, Gn) and
    // 64-wide rows (the rest).  Padding spreads the 16 rows an operand read or
    // a tile write touches over the banks; measured at the 2.7B shape (row
    // strides 72 / N + 8 before): 80 / N + 16 0.885 ms per backward, 80 / N + 8
    // 0.903, 88 / N + 8 0.935, 72 / N + 8 0.918.  With the float32 dy copy
    // (H32) the 64-wide rows keep 72 elements so that it still fits.
    static constexpr int kLdN = N + 16;
    static constexpr int kLdC = H32 ? kLd : kLd + 8;
    static constexpr int kLdF = kP2 + 4;   // row stride (floats) of the float32 dy copy (H32)
    static constexpr size_t kBytes =
        sizeof(u16) * (2 * static_cast<size_t>(kQ2) * kLdN + 2 * N * kLdC + 6 * kQ2 * kLdC) +
        (H32 ? sizeof(float) * kQ2 * kLdF : 0);
};

// The score tiles (u-tile, t-tile) with u >= t, and those above the diagonal,
// dealt to the wavefronts: wavefront w evaluates kLowerTile[w] and, for w < 2,
// kLowerTile[w + 8]; wavefronts 2..7 clear kUpperTile[w - 2].
__constant__ int2 kLowerTile[10] = {{0, 0}, {1, 0}, {1, 1}, {2, 0}, {2, 1}, {2, 2}, {3, 0}, {3, 1}, {3, 2}, {3, 3}};
__constant__ int2 kUpperTile[6] = {{0, 1}, {0, 2}, {0, 3}, {1, 2}, {1, 3}, {2, 3}};

// DIRECT: one head slice per group; dB and dC stored by this kernel (bf16).
template <int N, bool PACKED, bool H32, bool DIRECT>
// A_log and D come as separate read-only arguments so that their per-head
// values are scalar loads: read through the parameter block (whose other
// pointers the kernel writes through) they were vector loads, and the wait for
// them at every head's start also waited for all the memory operations
// before them, the previous head's gradient stores included.
__global__ __launch_bounds__(kT2) void k_bwd2_chunk(BwdParams p, const float* __restrict__ A_logp,
                                                    const float* __restrict__ Dp)
{
    constexpr int kLdN = ChunkSmem<N>::kLdN;
    constexpr int kLdF = ChunkSmem<N, H32>::kLdF;
    constexpr int kLd = ChunkSmem<N, H32>::kLdC;   // (this kernel's 64-wide row stride)
    constexpr int kNT = N / 16;             // n-tiles
    constexpr int kBW = N / 32;             // dB / dC tiles per wavefront
    extern __shared__ __attribute__((aligned(16))) u16 sm2[];
    u16* Bs = sm2;                      // 64 x kLdN  B   (row t, k = n)
    u16* BT = Bs + kQ2 * kLdN;          // N x kLd    B^T (row n, k = t)
    u16* CT = BT + N * kLd;             // N x kLd    C^T (row n, k = u)
    u16* xs = CT + N * kLd;             // 64 x kLd   x   (row t, k = p)
    u16* dys = xs + kQ2 * kLd;          // 64 x kLd   dy  (row u, k = p)
    u16* dyT = dys + kQ2 * kLd;         // 64 x kLd   dy^T (row p, k = u)
    u16* GsT = dyT + kQ2 * kLd;         // 64 x kLd   Gs^T (row t, k = u)
    u16* Rs = GsT + kQ2 * kLd;          // 64 x kLd   Rs  (row u, k = t)
    u16* RsT = Rs + kQ2 * kLd;          // 64 x kLd   Rs^T (row t, k = u)
    u16* GnS = RsT + kQ2 * kLd;         // 64 x kLdN  Gn  (row p, k = n), from Gn^T
    float* dyF = reinterpret_cast<float*>(GnS + kQ2 * kLdN);   // H32: 64 x kLdF dy in float32 (row u)
    // per-token factors, double-buffered by head parity (the per-token phase of
    // one head overlaps the next head's set-up)
    __shared__ float scs2[2][kQ2], sdt2[2][kQ2], seend2[2][kQ2], secs2[2][kQ2];
    __shared__ float rowp[kQ2][4], colp[kQ2][4], xdxp[kQ2][4], q2p[kQ2][4], dyxp[kQ2][4], q1p[kQ2][kNT];
    __shared__ float scr[8];

    const int64_t c = blockIdx.x, b = blockIdx.y;
    const HeadRange hr = head_range(p);
    // wavefront index, provably uniform: the tile tables below are read with
    // scalar loads, never vector loads whose wait would also wait for the
    // next head's inputs in flight
    const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane & 15, q = lane >> 4;
    int L0 = 0;
    int64_t t00 = 0;
    if constexpr (PACKED) {   // chunk c of the table; entries past its end add nothing to dA, dD
        if (c >= *p.vcount) {
            for (int64_t hh = hr.lo + tid; hh < hr.hi; hh += kT2) {
                p.dAp[hh * p.nC + c] = 0.f;
                p.dDp[hh * p.nC + c] = 0.f;
            }
            return;
        }
        const int4 e = p.vtab[c];
        L0 = e.y;
        t00 = e.x;
    } else {
        L0 = chunk_len2(p.T, c);
        t00 = b * p.T + c * kQ2;
    }
    const int L = L0;
    const int64_t t0 = t00;
    const u16* Bg = static_cast<const u16*>(p.B);
    const u16* Cg = static_cast<const u16*>(p.C);
    const u16* xg = static_cast<const u16*>(p.x);
    const u16* dyg = static_cast<const u16*>(p.dy);
    const float* dyg32 = static_cast<const float*>(p.dy);   // H32
    u16* dxg = static_cast<u16*>(p.dx);

    // B, B^T, C^T of the chunk
    for (int i = tid; i < kQ2 * N / 8; i += kT2) {
        const int s = i & 63, n0 = 8 * (i >> 6);   // consecutive lanes: consecutive tokens
        uint4 vb = make_uint4(0, 0, 0, 0), vc = vb;
        if (s < L) {
            const int64_t gi = ((t0 + s) * p.G + hr.g) * N + n0;
            vb = *reinterpret_cast<const uint4*>(Bg + gi);
            vc = *reinterpret_cast<const uint4*>(Cg + gi);
        }
        *reinterpret_cast<uint4*>(Bs + s * kLdN + n0) = vb;
        const uint32_t eb[4] = {vb.x, vb.y, vb.z, vb.w}, ec[4] = {vc.x, vc.y, vc.z, vc.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            BT[(n0 + 2 * e) * kLd + s] = static_cast<u16>(eb[e]);
            BT[(n0 + 2 * e + 1) * kLd + s] = static_cast<u16>(eb[e] >> 16);
            CT[(n0 + 2 * e) * kLd + s] = static_cast<u16>(ec[e]);
            CT[(n0 + 2 * e + 1) * kLd + s] = static_cast<u16>(ec[e] >> 16);
        }
    }
    __syncthreads();

    // G0 = C B^T on this wavefront's score tiles (C rows straight from global memory)
    const int ntile = w < 2 ? 2 : 1;
    f32x4_t g0[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        g0[k] = zero4();
        if (k < ntile) {
            const int2 tl = kLowerTile[w + 8 * k];
            const int u = 16 * tl.x + r;
            const int64_t crow = ((t0 + (u < L ? u : 0)) * p.G + hr.g) * N;
#pragma unroll
            for (int ks = 0; ks < N / 32; ++ks) {
                uint4 a = *reinterpret_cast<const uint4*>(Cg + crow + ks * 32 + 8 * q);
                if (u >= L) a = make_uint4(0, 0, 0, 0);
                g0[k] = mma(a, ldfrag(Bs, kLdN, 16 * tl.y + r, ks, lane), g0[k]);
            }
        }
    }

    f32x4_t dBacc[kBW], dCacc[kBW];
#pragma unroll
    for (int j = 0; j < kBW; ++j) dBacc[j] = dCacc[j] = zero4();

    // one head's inputs, fetched a head ahead: dt (wavefront 0, lane = token)
    // and one 8-wide piece of x and of dy per thread (token s_me = lane)
    const int s_me = lane, p0_me = 8 * w;   // token = lane, 8 p values per wavefront
    uint32_t pdt = 0;   // raw bits (see load_dt_raw)
    uint4 px = make_uint4(0, 0, 0, 0), pd = px;
    float4 pf0 = make_float4(0.f, 0.f, 0.f, 0.f), pf1 = pf0;   // H32: dy in float32
    const auto fetch = [&](int64_t h) {
        if (w == 0) pdt = lane < L ? load_dt_raw<H32>(p.dt, (t0 + lane) * p.H + h) : 0u;
        px = pd = make_uint4(0, 0, 0, 0);
        pf0 = pf1 = make_float4(0.f, 0.f, 0.f, 0.f);
        if (s_me < L) {
            const int64_t gi = ((t0 + s_me) * p.H + h) * kP2 + p0_me;
            px = *reinterpret_cast<const uint4*>(xg + gi);
            if constexpr (H32) {
                pf0 = *reinterpret_cast<const float4*>(dyg32 + gi);
                pf1 = *reinterpret_cast<const float4*>(dyg32 + gi + 4);
            } else {
                pd = *reinterpret_cast<const uint4*>(dyg + gi);
            }
        }
    };
    fetch(hr.lo);

    for (int64_t h = hr.lo; h < hr.hi; ++h) {
        const int64_t bh = b * p.H + h;
        const int64_t sbase = ((b * p.nC + c) * p.H + h) * kP2 * N;
        const u16* GnT = reinterpret_cast<const u16*>(p.gnT) + sbase;   // n x p
        const u16* HinT = reinterpret_cast<const u16*>(p.hin) + sbase;  // n x p
        const float Ah = -expf(A_logp[h]);
        const float Dh = Dp ? Dp[h] : 0.f;
        const int hb = static_cast<int>((h - hr.lo) & 1);
        float* const scs = scs2[hb];
        float* const sdt = sdt2[hb];
        float* const seend = seend2[hb];
        float* const secs = secs2[hb];

        // this wavefront's state fragments (issued first: they come from HBM)
        const int pw = w >> 1;                       // p-tile of dX^T
        uint4 gpc[N / 64], gntf[2], hinf[2];   // pieces of Gn^T for GnS; operand fragments
#pragma unroll
        for (int k = 0; k < N / 64; ++k) {
            // piece (row n = pc % N, p = 8 (pc / N) ..): consecutive lanes, consecutive rows
            const int pc = tid + kT2 * k, nn = pc % N, p0 = 8 * (pc / N);
            gpc[k] = reinterpret_cast<const uint4*>(GnT)[nn * (kP2 / 8) + p0 / 8];
        }
        {
            const int nt = (w * kBW) >> 2;   // this wavefront's n-tile of dB^T / dC^T (one per wavefront)
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                gntf[ks] = ldfrag_g(GnT, kP2, 16 * nt + r, ks, lane);
                hinf[ks] = ldfrag_g(HinT, kP2, 16 * nt + r, ks, lane);
            }
        }
        // this head's x, dy (fetched during the previous head) into shared memory
        if constexpr (H32) {   // the operand copies in bf16, dy also kept in float32
            pd = make_uint4(pack2(pf0.x, pf0.y), pack2(pf0.z, pf0.w), pack2(pf1.x, pf1.y), pack2(pf1.z, pf1.w));
            *reinterpret_cast<float4*>(dyF + s_me * kLdF + p0_me) = pf0;
            *reinterpret_cast<float4*>(dyF + s_me * kLdF + p0_me + 4) = pf1;
        }
        *reinterpret_cast<uint4*>(xs + s_me * kLd + p0_me) = px;
        *reinterpret_cast<uint4*>(dys + s_me * kLd + p0_me) = pd;
        {
            const uint32_t ed[4] = {pd.x, pd.y, pd.z, pd.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                dyT[(p0_me + 2 * e) * kLd + s_me] = static_cast<u16>(ed[e]);
                dyT[(p0_me + 2 * e + 1) * kLd + s_me] = static_cast<u16>(ed[e] >> 16);
            }
        }
        if (w == 0) {
            // cumsum of dt*A (log2 units) and the per-token factors
            const float A2 = Ah * kLog2e;
            const float dtv = dt_of_raw<H32>(pdt);
            const float cs = wave_scan(dtv * A2);
            const float csend = lane_value(cs, L - 1);
            scs[lane] = cs;
            sdt[lane] = dtv;
            seend[lane] = lane < L ? exp2f(csend - cs) : 0.f;
            secs[lane] = lane < L ? exp2f(cs) : 0.f;
        }
        if (h + 1 < hr.hi) fetch(h + 1);
        __syncthreads();   // (1) per-head inputs in place

        // --- score tiles: R0 = dy x^T (then dt_t), Gs, Rs, l and their sums
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            if (k < ntile) {
                const int2 tl = kLowerTile[w + 8 * k];
                f32x4_t acc = zero4();
#pragma unroll
                for (int ks = 0; ks < 2; ++ks)
                    acc = mma(ldfrag(dys, kLd, 16 * tl.x + r, ks, lane), ldfrag(xs, kLd, 16 * tl.y + r, ks, lane),
                              acc);
                const int t = 16 * tl.y + r;
                const float dtt = sdt[t], cst = scs[t];
                float gs[4], rs[4], colsum = 0.f;
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int u = 16 * tl.x + 4 * q + v;
                    float gv = 0.f, rv = 0.f, lv = 0.f;
                    if (u >= t && u < L) {
                        const float e = exp2f(scs[u] - cst);
                        const float r0 = acc[v] * dtt;
                        gv = e * g0[k][v];
                        rv = e * r0;
                        lv = gv * r0;
                    }
                    gs[v] = gv;
                    rs[v] = rv;
                    colsum += lv;
                    // row sum of l over the tile's 16 columns t
                    const float rsum = row_sum16(lv);
                    if (r == 0) rowp[16 * tl.x + 4 * q + v][tl.y] = rsum;
                }
                colsum = col_sum4(colsum);
                if (q == 0) colp[t][tl.x] = colsum;
                const int u0 = 16 * tl.x + 4 * q;
                *reinterpret_cast<uint2*>(GsT + t * kLd + u0) = make_uint2(pack2(gs[0], gs[1]), pack2(gs[2], gs[3]));
                *reinterpret_cast<uint2*>(RsT + t * kLd + u0) = make_uint2(pack2(rs[0], rs[1]), pack2(rs[2], rs[3]));
#pragma unroll
                for (int v = 0; v < 4; ++v) Rs[(u0 + v) * kLd + t] = static_cast<u16>(bf16_bits(rs[v]));
            }
        }
        if (w >= 2) {
            const int2 tl = kUpperTile[w - 2];
            const int t = 16 * tl.y + r, u0 = 16 * tl.x + 4 * q;
            *reinterpret_cast<uint2*>(GsT + t * kLd + u0) = make_uint2(0, 0);
            *reinterpret_cast<uint2*>(RsT + t * kLd + u0) = make_uint2(0, 0);
#pragma unroll
            for (int v = 0; v < 4; ++v) Rs[(u0 + v) * kLd + t] = 0;
            if (r == 0)
#pragma unroll
                for (int v = 0; v < 4; ++v) rowp[u0 + v][tl.y] = 0.f;
            if (q == 0) colp[t][tl.x] = 0.f;
        }
        // Gn (p x n) into shared memory from the pieces of Gn^T
#pragma unroll
        for (int k = 0; k < N / 64; ++k) {
            const int pc = tid + kT2 * k, nn = pc % N, p0 = 8 * (pc / N);
            const uint32_t eg[4] = {gpc[k].x, gpc[k].y, gpc[k].z, gpc[k].w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                GnS[(p0 + 2 * e) * kLdN + nn] = static_cast<u16>(eg[e]);
                GnS[(p0 + 2 * e + 1) * kLdN + nn] = static_cast<u16>(eg[e] >> 16);
            }
        }
        __syncthreads();   // (2) score tiles, their sums and Gn in place

        // --- dX~^T (p x t): dy^T Gs + e(end,t) Gn B^T; dx, and per-token sums
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int tt = 2 * (w & 1) + j;
            f32x4_t ai = zero4(), ag = zero4();
#pragma unroll
            for (int ks = 0; ks < 2; ++ks)
                ai = mma(ldfrag(dyT, kLd, 16 * pw + r, ks, lane), ldfrag(GsT, kLd, 16 * tt + r, ks, lane), ai);
#pragma unroll
            for (int ks = 0; ks < N / 32; ++ks)
                ag = mma(ldfrag(GnS, kLdN, 16 * pw + r, ks, lane), ldfrag(Bs, kLdN, 16 * tt + r, ks, lane), ag);
            const int t = 16 * tt + r, p0 = 16 * pw + 4 * q;
            const float ee = seend[t], dtt = sdt[t];
            const uint2 xv = *reinterpret_cast<const uint2*>(xs + t * kLd + p0);
            const float xf[4] = {lo_f(xv.x), hi_f(xv.x), lo_f(xv.y), hi_f(xv.y)};
            float df[4];
            if constexpr (H32) {
                const float4 d4 = *reinterpret_cast<const float4*>(dyF + t * kLdF + p0);
                df[0] = d4.x; df[1] = d4.y; df[2] = d4.z; df[3] = d4.w;
            } else {
                const uint2 dv = *reinterpret_cast<const uint2*>(dys + t * kLd + p0);
                df[0] = lo_f(dv.x); df[1] = hi_f(dv.x); df[2] = lo_f(dv.y); df[3] = hi_f(dv.y);
            }
            float dx[4], sxd = 0.f, sxg = 0.f, sdx = 0.f;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const float dX = fmaf(ee, ag[v], ai[v]);
                dx[v] = fmaf(dtt, dX, Dh * df[v]);
                sxd = fmaf(xf[v], dX, sxd);
                sxg = fmaf(xf[v], ag[v], sxg);
                sdx = fmaf(df[v], xf[v], sdx);
            }
            if (t < L)
                *reinterpret_cast<uint2*>(dxg + (t0 + t) * p.H * kP2 + h * kP2 + p0) =
                    make_uint2(pack2(dx[0], dx[1]), pack2(dx[2], dx[3]));
            sxd = col_sum4(sxd);
            sxg = col_sum4(sxg);
            sdx = col_sum4(sdx);
            if (q == 0) {
                xdxp[t][pw] = sxd;
                q2p[t][pw] = sxg;
                dyxp[t][pw] = sdx;
            }
        }

        // --- dB^T (n x t) += C^T Rs + e(end,t) dt_t Gn^T x^T
#pragma unroll
        for (int j = 0; j < kBW; ++j) {
            const int idx = w * kBW + j, nt = idx >> 2, tt = idx & 3;
            f32x4_t bi = zero4(), bx = zero4();
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                bi = mma(ldfrag(CT, kLd, 16 * nt + r, ks, lane), ldfrag(RsT, kLd, 16 * tt + r, ks, lane), bi);
                bx = mma(gntf[ks], ldfrag(xs, kLd, 16 * tt + r, ks, lane), bx);
            }
            const int t = 16 * tt + r;
            const float fb = seend[t] * sdt[t];
#pragma unroll
            for (int v = 0; v < 4; ++v) dBacc[j][v] += fmaf(fb, bx[v], bi[v]);
        }
        // --- dC^T (n x u) += B^T Rs^T + exp(cs_u) h_in^T dy^T, and dy_u . (h_in C_u)
#pragma unroll
        for (int j = 0; j < kBW; ++j) {
            const int idx = w * kBW + j, nt = idx >> 2, tt = idx & 3;
            f32x4_t ci = zero4(), ch = zero4();
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                ci = mma(ldfrag(BT, kLd, 16 * nt + r, ks, lane), ldfrag(Rs, kLd, 16 * tt + r, ks, lane), ci);
                ch = mma(hinf[ks], ldfrag(dys, kLd, 16 * tt + r, ks, lane), ch);
            }
            const int t = 16 * tt + r;
            const float fc = secs[t];
            float q1 = 0.f;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                dCacc[j][v] += fmaf(fc, ch[v], ci[v]);
                q1 = fmaf(bf(CT[(16 * nt + 4 * q + v) * kLd + t]), ch[v], q1);
            }
            q1 = col_sum4(q1);
            if (q == 0) q1p[t][nt] = q1;
        }

        {
            // <Gn, h_in> from this wavefront's fragments of Gn^T and h_in^T (one
            // n-tile; with dstate 64 two wavefronts hold each tile, the even one counts it)
            float gh = 0.f;
            if (kBW == 4 || (w & 1) == 0) {
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) {
                    const uint32_t ea[4] = {gntf[ks].x, gntf[ks].y, gntf[ks].z, gntf[ks].w};
                    const uint32_t ez[4] = {hinf[ks].x, hinf[ks].y, hinf[ks].z, hinf[ks].w};
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        gh = fmaf(lo_f(ea[e]), lo_f(ez[e]), fmaf(hi_f(ea[e]), hi_f(ez[e]), gh));
                }
            }
            gh = wave_sum(gh);
            if (lane == 0) scr[w] = gh;
        }
        __syncthreads();   // (3) per-token partial sums in place

        // --- per token (wavefront 1; lane k holds token t = 63 - k, so that a
        // prefix sum over lanes is a suffix sum over tokens): dcs, then the decay
        // gradients.  The other wavefronts go on to the next head's set-up
        // meanwhile; what they write there (inputs, the other buffer of
        // per-token factors) this does not read, and the partial sums are
        // rewritten only after the next barrier (1).
        if (w == 1) {
            const int t = kQ2 - 1 - lane;
            const bool in = t < L;
            float s2 = 0.f, row = 0.f, col = 0.f, s1 = 0.f, xd = 0.f, dyx = 0.f;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                s2 += q2p[t][k];
                row += rowp[t][k];
                col += colp[t][k];
                xd += xdxp[t][k];
                dyx += dyxp[t][k];
            }
#pragma unroll
            for (int k = 0; k < kNT; ++k) s1 += q1p[t][k];
            const float q2 = in ? sdt[t] * s2 : 0.f;   // X~_t . (Gn B_t)
            const float ghs = ((scr[0] + scr[1]) + (scr[2] + scr[3])) + ((scr[4] + scr[5]) + (scr[6] + scr[7]));
            const float hsum = wave_sum(seend[t] * q2);
            float dcs = in ? row - col + secs[t] * s1 - seend[t] * q2 : 0.f;
            if (t == L - 1) dcs += secs[t] * ghs + hsum;   // <Gn, h_out>
            const float da = wave_scan(dcs);   // over tokens t' >= t
            if (in) {
                const float g = fmaf(Ah, da, xd);
                if constexpr (H32)
                    static_cast<float*>(p.ddt)[(t0 + t) * p.H + h] = g;
                else
                    static_cast<u16*>(p.ddt)[(t0 + t) * p.H + h] = static_cast<u16>(bf16_bits(g));
            }
            const float sa = wave_sum(in ? sdt[t] * da : 0.f);
            const float sd = wave_sum(in ? dyx : 0.f);
            if (lane == 0) {
                p.dAp[bh * p.nC + c] = sa;
                p.dDp[bh * p.nC + c] = sd;
            }
        }
    }

    // this slice's dB and dC for the chunk: lane holds n = 16 nt + 4 q + v, t = 16 tt + r.
    // With one slice per group these sums are the gradients: rounded here to
    // bf16 (nearest even, as the reduction over slices rounds them) and stored
    // in place, and the launch skips that reduction (bc_direct).
#pragma unroll
    for (int j = 0; j < kBW; ++j) {
        const int idx = w * kBW + j, nt = idx >> 2, tt = idx & 3;
        const int t = 16 * tt + r;
        if (t < L) {
            if constexpr (DIRECT) {
                const int64_t o = ((t0 + t) * p.G + hr.g) * N + 16 * nt + 4 * q;
                *reinterpret_cast<uint2*>(static_cast<u16*>(p.dB) + o) =
                    make_uint2(rne_pair(dBacc[j][0], dBacc[j][1]), rne_pair(dBacc[j][2], dBacc[j][3]));
                *reinterpret_cast<uint2*>(static_cast<u16*>(p.dC) + o) =
                    make_uint2(rne_pair(dCacc[j][0], dCacc[j][1]), rne_pair(dCacc[j][2], dCacc[j][3]));
            } else {
                const int64_t o = ((hr.slice * p.b * p.T + t0 + t) * p.G + hr.g) * N + 16 * nt + 4 * q;
                *reinterpret_cast<float4*>(p.dBp + o) =
                    make_float4(dBacc[j][0], dBacc[j][1], dBacc[j][2], dBacc[j][3]);
                *reinterpret_cast<float4*>(p.dCp + o) =
                    make_float4(dCacc[j][0], dCacc[j][1], dCacc[j][2], dCacc[j][3]);
            }
        }
    }
}

template <int N, bool PACKED, bool H32, bool DIRECT>
hipError_t launch_chunk(const BwdParams& p, dim3 grid, size_t sm, hipStream_t st)
{
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_bwd2_chunk<N, PACKED, H32, DIRECT>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(sm));
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((k_bwd2_chunk<N, PACKED, H32, DIRECT>), grid, dim3(kT2), sm, st, p, p.A_log, p.D);
    return hipGetLastError();
}

template <int N>
hipError_t launch_fast(const BwdParams& params, hipStream_t st, hipEvent_t ev0, hipEvent_t ev1)
{
    BwdParams p = params;
    p.bc_direct = p.S == 1 && reinterpret_cast<uintptr_t>(p.dB) % 8 == 0 && reinterpret_cast<uintptr_t>(p.dC) % 8 == 0;
    const bool packed = p.vtab != nullptr, h32 = p.h32 != 0, direct = p.bc_direct != 0;
    if (packed && h32) return hipErrorInvalidValue;   // float32 handoffs: plain rows only
    const size_t sm_chunk = h32 ? ChunkSmem<N, true>::kBytes : ChunkSmem<N>::kBytes;
    hipError_t e;
    if (packed)   // one workgroup per (sequence, head) and direction
        hipLaunchKernelGGL((k_bwd2_pass<N, true, false>), dim3(static_cast<unsigned>(p.nseq * p.H), 2), dim3(kPassT),
                           0, st, p);
    else if (h32)
        hipLaunchKernelGGL((k_bwd2_pass<N, false, true>), dim3(static_cast<unsigned>(p.b * p.H), 2), dim3(kPassT), 0,
                           st, p);
    else
        hipLaunchKernelGGL((k_bwd2_pass<N, false, false>), dim3(static_cast<unsigned>(p.b * p.H), 2), dim3(kPassT), 0,
                           st, p);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (ev0 && (e = hipEventRecord(ev0, st)) != hipSuccess) return e;
    const dim3 grid(static_cast<unsigned>(p.nC), static_cast<unsigned>(p.b), static_cast<unsigned>(p.G * p.S));
    if (packed)
        e = direct ? launch_chunk<N, true, false, true>(p, grid, sm_chunk, st)
                   : launch_chunk<N, true, false, false>(p, grid, sm_chunk, st);
    else if (h32)
        e = direct ? launch_chunk<N, false, true, true>(p, grid, sm_chunk, st)
                   : launch_chunk<N, false, true, false>(p, grid, sm_chunk, st);
    else
        e = direct ? launch_chunk<N, false, false, true>(p, grid, sm_chunk, st)
                   : launch_chunk<N, false, false, false>(p, grid, sm_chunk, st);
    if (e != hipSuccess) return e;
    if (ev1 && (e = hipEventRecord(ev1, st)) != hipSuccess) return e;
    return launch_backward_reduce(p, true, st, !direct);
}

}  // namespace

bool bwd_fast_supported(bool bf16, int64_t P, int64_t N) { return bf16 && P == kP2 && (N == 64 || N == 128); }

hipError_t launch_backward_fast(const BwdParams& p, hipStream_t stream, hipEvent_t ev_begin, hipEvent_t ev_end)
{
    return p.N == 64 ? launch_fast<64>(p, stream, ev_begin, ev_end) : launch_fast<128>(p, stream, ev_begin, ev_end);
}

}  // namespace ssd
