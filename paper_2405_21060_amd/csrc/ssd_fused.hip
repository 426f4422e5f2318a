// Fused SSD forward for the Mamba-2 layer shapes: bf16 activations, head
// dimension P = 64, state N in {64, 128}, chunk Q = 256, no packed rows.
//
// Two launches per call.
//
// k_fused_prep, one workgroup per (batch, chunk, group):
//   * step 1 for every head of the group: a = dt*A, chunk-local inclusive
//     cumsum in log2 units (cs2), written per (batch, head, chunk) together
//     with dt itself, both as float32 rows of Q (coalesced for the main kernel);
//   * B^T of the chunk (N x Q, bf16), the operand layout the chunk-state
//     contraction needs (contraction over tokens);
//   * the Gram matrix C B^T of the chunk (Section 5, eq. ssm-quad: G = C B^T),
//     only its causal 16x16 tiles, stored in the exact per-lane accumulator
//     layout in which the main kernel's wavefronts hold them.
//
// k_fused_main, one workgroup (8 wavefronts) per (chunk, batch, group of HG
// heads), ordered chunk-major through a ticket counter:
//   * the chunk's Gram tiles are streamed from L2 in their per-lane layout;
//     B^T is staged in LDS once, x^T (P x Q) per head;
//   * right factor (Section 6.2): S = sum_s dt_s exp(cs_end - cs_s) x_s B_s^T on
//     the matrix cores;
//   * diagonal block (Section 6.1): Y^T = x^T (L o G)^T dt, the mask applied to
//     the Gram fragments in registers and fed straight back into the matrix cores
//     (accumulator layout -> operand layout by permuting the contraction index);
//   * centre factor (Section 6.2, scalar scan of Appendix B, sequential
//     chunk-to-chunk state passing): wait for the state entering the chunk,
//     publish h_c = exp(cs_end) h_{c-1} + S for the next chunk;
//   * left factor: Y^T += exp(cs_t) (h_{c-1} C_t^T), then + D x, stored bf16.
//
// Cross-workgroup state passing.  States go through a two-slot ring per
// (batch, head); h_c is written with device-coherent (sc1) stores, the stores
// are drained (s_waitcnt vmcnt(0)), then a per-(batch, head, chunk) flag is
// set with a device-coherent store.  The successor polls the flag and reads
// the state with device-coherent loads.  No cache-wide writeback/invalidate is
// needed because every access to shared data is device-coherent.  Workgroups
// take their work item from a ticket counter in dispatch order, so a
// workgroup only ever waits on an item already owned by a running or finished
// workgroup; the wait is additionally bounded (a timeout sets an error word).
// Two ring slots suffice: chunk c+2 overwrites the slot of chunk c only after
// reading the state of chunk c+1, which chunk c+1 published only after it had
// read (consumed) the state of chunk c.
#include "ssd_device.h"
#include "ssd_internal.h"

namespace ssd {
namespace {

constexpr int kQ = 256;                       // chunk length
constexpr int kNQ = kQ / 16;                  // 16-token strips per chunk
constexpr int kTiles = kNQ * (kNQ + 1) / 2;   // causal 16x16 tiles (s-tile <= t-tile)
constexpr int kP = 64;                        // head dimension
constexpr int kWaves = 8;
constexpr int kMainThreads = kWaves * 64;
constexpr int kPrepThreads = 256;
constexpr int kRowPad = 8;                    // bf16 elements of padding per LDS row
constexpr int kQS = kQ + kRowPad;             // LDS row stride of token-major rows
constexpr long long kSpinLimit = 1LL << 22;   // polls (with s_sleep) before giving up

typedef unsigned short u16;
typedef uint32_t u32;
typedef u32 uint4_t __attribute__((ext_vector_type(4)));

struct U16x8 {
    u16 v[8];
};

__device__ __forceinline__ float bf(u16 u) { return __uint_as_float(static_cast<u32>(u) << 16); }

__device__ __forceinline__ u16 to_bf16(float f)
{
    u32 u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return static_cast<u16>(u >> 16);
}

__device__ __forceinline__ bf16x8_t pack8(const float* f)
{
    bf16x8_t r;
#pragma unroll
    for (int e = 0; e < 8; ++e) r[e] = static_cast<__bf16>(f[e]);
    return r;
}

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 v)
{
    return __builtin_bit_cast(bf16x8_t, v);
}

__device__ __forceinline__ f32x4_t mfma(bf16x8_t a, bf16x8_t b, f32x4_t c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Drain this wavefront's outstanding vector-memory operations.
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

__device__ __forceinline__ float ld_coherent(const float* p)
{
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void st_coherent(float* p, float v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Causal tile index of (s-tile j, t-tile i), j <= i.
__device__ __forceinline__ int tile_index(int i, int j) { return i * (i + 1) / 2 + j; }

// ---------------------------------------------------------------------------
// prep
// ---------------------------------------------------------------------------
constexpr int kPrepParts = 8;   // workgroups per (batch, chunk, group)

template <int N>
__global__ __launch_bounds__(kPrepThreads) void k_fused_prep(FusedParams p)
{
    const int c = blockIdx.x;
    const int b = static_cast<int>(blockIdx.y / p.G), g = static_cast<int>(blockIdx.y % p.G);
    const int part = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, r = lane & 15, lg = lane >> 4;
    const int64_t c0 = static_cast<int64_t>(c) * kQ;
    const int L = static_cast<int>(kQ < p.T - c0 ? kQ : p.T - c0);
    const int hpg = static_cast<int>(p.H / p.G);
    const u16* dtp = static_cast<const u16*>(p.dt);
    const u16* Bp = static_cast<const u16*>(p.B);
    const u16* Cp = static_cast<const u16*>(p.C);

    // flags of this (batch, chunk) and group, and the ticket counter
    if (part == 0) {
        for (int hh = tid; hh < hpg; hh += kPrepThreads)
            p.flags[(static_cast<int64_t>(b) * p.H + g * hpg + hh) * p.nC + c] = 0;
        if (blockIdx.x == 0 && blockIdx.y == 0 && tid == 0) {
            p.ticket[0] = 0;
            p.ticket[1] = 0;  // error word: set when a state wait times out
        }
    }

    // step 1 for the heads of this part: one wavefront per head, 4 tokens per lane
    for (int hh = part * 4 + wave; hh < hpg; hh += kPrepParts * 4) {
        const int h = g * hpg + hh;
        const float A2 = -expf(p.A_log[h]) * kLog2e;
        float d[4], a[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int t = 4 * lane + k;
            d[k] = (t < L) ? bf(dtp[(b * p.T + c0 + t) * p.H + h]) : 0.f;
            a[k] = d[k] * A2;
        }
        a[1] += a[0];
        a[2] += a[1];
        a[3] += a[2];
        float incl = a[3];
#pragma unroll
        for (int s = 1; s < 64; s <<= 1) {
            const float o = __shfl_up(incl, s, 64);
            if (lane >= s) incl += o;
        }
        const float excl = incl - a[3];
        const int64_t row = ((static_cast<int64_t>(b) * p.H + h) * p.nC + c) * kQ + 4 * lane;
        *reinterpret_cast<float4*>(p.cs2 + row) = make_float4(a[0] + excl, a[1] + excl, a[2] + excl, a[3] + excl);
        *reinterpret_cast<float4*>(p.dtT + row) = make_float4(d[0], d[1], d[2], d[3]);
    }

    // B^T of the chunk, rows n of this part: lanes walk n (coalesced row reads of B)
    u16* bt = p.BT + ((static_cast<int64_t>(b) * p.G + g) * p.nC + c) * N * kQ;
    constexpr int kBtItems = N * (kQ / 8) / kPrepParts;
    for (int idx = tid; idx < kBtItems; idx += kPrepThreads) {
        const int gi = part * kBtItems + idx;
        const int n = gi % N, so = gi / N;
        U16x8 v;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int s = 8 * so + e;
            v.v[e] = (s < L) ? Bp[((b * p.T + c0 + s) * p.G + g) * N + n] : static_cast<u16>(0);
        }
        *reinterpret_cast<uint4*>(bt + static_cast<int64_t>(n) * kQ + 8 * so) = __builtin_bit_cast(uint4, v);
    }

    // Gram tiles G^T[s][t] = sum_n B_s[n] C_t[n] (bf16), accumulator layout per lane
    u16* gram = p.gram + ((static_cast<int64_t>(b) * p.G + g) * p.nC + c) * kTiles * 256;
    for (int ti = part * 4 + wave; ti < kTiles; ti += kPrepParts * 4) {
        int i = 0;
        while ((i + 1) * (i + 2) / 2 <= ti) ++i;
        const int j = ti - i * (i + 1) / 2;
        const int s = 16 * j + r, t = 16 * i + r;
        f32x4_t acc = zero4();
#pragma unroll
        for (int k0 = 0; k0 < N; k0 += 32) {
            uint4 va = make_uint4(0, 0, 0, 0), vb = make_uint4(0, 0, 0, 0);
            if (s < L) va = *reinterpret_cast<const uint4*>(Bp + ((b * p.T + c0 + s) * p.G + g) * N + k0 + 8 * lg);
            if (t < L) vb = *reinterpret_cast<const uint4*>(Cp + ((b * p.T + c0 + t) * p.G + g) * N + k0 + 8 * lg);
            acc = mfma(as_bf16x8(va), as_bf16x8(vb), acc);
        }
        uint2 packed;
        packed.x = static_cast<u32>(to_bf16(acc[0])) | (static_cast<u32>(to_bf16(acc[1])) << 16);
        packed.y = static_cast<u32>(to_bf16(acc[2])) | (static_cast<u32>(to_bf16(acc[3])) << 16);
        *reinterpret_cast<uint2*>(gram + (static_cast<int64_t>(ti) * 64 + lane) * 4) = packed;
    }
}

// ---------------------------------------------------------------------------
// main
// ---------------------------------------------------------------------------
template <int N>
struct MainSmem {
    u16 GR[kTiles * 256];     // Gram tiles of the chunk: [tile][lane][4] bf16
    u16 XT[kP * kQS];         // x^T (P x Q) of the current head
    u16 XW[kP * kQS];         // x^T * w (P x Q); after the right factor: bf16 state (P x (N+8))
    float cs[kQ];             // cs2 of the current head
    float vf[kQ];             // dt_s exp2(cs2[tile end] - cs2_s)
    float w[kQ];              // dt_s exp2(cs2[Q-1] - cs2_s)
    float dt[kQ];
    int ticket;
};

// One K-step (32 tokens: s-tiles j0, j0+1) of the diagonal block for one
// 16-token strip: the masked Gram values become the B operand (contraction
// index permuted to the accumulator layout: slot e<4 -> s = 16 j0 + 4 lg + e,
// slot e>=4 -> s = 16 (j0+1) + 4 lg + e - 4), x^T rows the A operand.
// Off-diagonal tiles factor the mask as exp2(cs_t - cs_end(j)) * exp2(cs_end(j) - cs_s),
// both factors <= 1; the diagonal tile takes exp2(cs_t - cs_s) directly.
__device__ __forceinline__ void diag_step(const u16* XT, const float* cs, const float* vf,
                                          const float* dt, uint2 g0, uint2 g1, int j0, int strip,
                                          int t, float cst, int r, int lg, f32x4_t* y)
{
    float mv[8];
#pragma unroll
    for (int half = 0; half < 2; ++half) {
        const int j = j0 + half;
        const uint2 gp = half ? g1 : g0;
        const float gv[4] = {__uint_as_float(gp.x << 16), __uint_as_float(gp.x & 0xFFFF0000u),
                             __uint_as_float(gp.y << 16), __uint_as_float(gp.y & 0xFFFF0000u)};
        const int sb = 16 * j + 4 * lg;
        if (j < strip) {
            const float u = __builtin_amdgcn_exp2f(cst - cs[16 * j + 15]);
            const float4 vf4 = *reinterpret_cast<const float4*>(&vf[sb]);
            mv[4 * half + 0] = gv[0] * (u * vf4.x);
            mv[4 * half + 1] = gv[1] * (u * vf4.y);
            mv[4 * half + 2] = gv[2] * (u * vf4.z);
            mv[4 * half + 3] = gv[3] * (u * vf4.w);
        } else if (j == strip) {
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int s = sb + v;
                mv[4 * half + v] = (s <= t) ? gv[v] * (__builtin_amdgcn_exp2f(cst - cs[s]) * dt[s]) : 0.f;
            }
        } else {
#pragma unroll
            for (int v = 0; v < 4; ++v) mv[4 * half + v] = 0.f;
        }
    }
    const bf16x8_t bop = pack8(mv);
    const int sa = 16 * j0 + 4 * lg;
#pragma unroll
    for (int pt = 0; pt < 4; ++pt) {
        const u16* row = XT + (16 * pt + r) * kQS;
        const uint2 lo = *reinterpret_cast<const uint2*>(row + sa);
        const uint2 hi = *reinterpret_cast<const uint2*>(row + sa + 16);
        y[pt] = mfma(as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y)), bop, y[pt]);
    }
}

// All K-steps of the diagonal block for one strip (Gram tiles from LDS).
__device__ __forceinline__ void strip_diag(const u16* XT, const float* cs, const float* vf,
                                           const float* dt, const u16* GR, int strip,
                                           int r, int lg, int lane, f32x4_t* y)
{
    const int t = 16 * strip + r;
    const float cst = cs[t];
    const uint2* gt = reinterpret_cast<const uint2*>(GR) + tile_index(strip, 0) * 64 + lane;
    const int nsteps = strip / 2 + 1;
#pragma unroll 2
    for (int m = 0; m < nsteps; ++m) {
        const int j0 = 2 * m;
        const uint2 g0 = gt[j0 * 64];
        const uint2 g1 = (j0 + 1 <= strip) ? gt[(j0 + 1) * 64] : make_uint2(0, 0);
        diag_step(XT, cs, vf, dt, g0, g1, j0, strip, t, cst, r, lg, y);
    }
}

// x of one head: XV vectors of 8 bf16 per thread (token s, features p0..p0+7)
#define SSD_LOAD_X(hh)                                                                          \
    _Pragma("unroll") for (int k_ = 0; k_ < XV; ++k_) {                                         \
        const int vi_ = tid + kMainThreads * k_;                                                \
        const int s_ = vi_ >> 3, p0_ = (vi_ & 7) * 8;                                           \
        xr[k_] = make_uint4(0, 0, 0, 0);                                                        \
        if (s_ < L)                                                                             \
            xr[k_] = *reinterpret_cast<const uint4*>(xp + ((b * p.T + c0 + s_) * p.H + (hh)) * kP + p0_); \
    }
// x^T and (x * w)^T of one head into LDS (needs sm.w of that head)
#define SSD_STORE_X()                                                                           \
    _Pragma("unroll") for (int k_ = 0; k_ < XV; ++k_) {                                         \
        const int vi_ = tid + kMainThreads * k_;                                                \
        const int s_ = vi_ >> 3, p0_ = (vi_ & 7) * 8;                                           \
        const U16x8 v_ = __builtin_bit_cast(U16x8, xr[k_]);                                     \
        const float ws_ = sm.w[s_];                                                             \
        u16* xt_ = sm.XT + p0_ * kQS + s_;                                                      \
        u16* xw_ = sm.XW + p0_ * kQS + s_;                                                      \
        _Pragma("unroll") for (int e_ = 0; e_ < 8; ++e_) {                                      \
            xt_[e_ * kQS] = v_.v[e_];                                                           \
            xw_[e_ * kQS] = to_bf16(bf(v_.v[e_]) * ws_);                                        \
        }                                                                                       \
    }
#define SSD_LOAD_SCALARS(hh)                                                                    \
    if (tid < kQ) {                                                                             \
        const int64_t row_ = ((static_cast<int64_t>(b) * p.H + (hh)) * p.nC + c) * kQ;          \
        csr = p.cs2[row_ + tid];                                                                \
        dtr = p.dtT[row_ + tid];                                                                \
    }
// scalars of one head into LDS, then the per-token weights (two barriers)
#define SSD_STORE_SCALARS()                                                                     \
    {                                                                                           \
        if (tid < kQ) {                                                                         \
            sm.cs[tid] = csr;                                                                   \
            sm.dt[tid] = dtr;                                                                   \
        }                                                                                       \
        __syncthreads();                                                                        \
        if (tid < kQ) {                                                                         \
            sm.vf[tid] = dtr * exp2f(sm.cs[tid | 15] - csr);                                    \
            sm.w[tid] = dtr * exp2f(sm.cs[kQ - 1] - csr);                                       \
        }                                                                                       \
        __syncthreads();                                                                        \
    }

template <int N>
__global__ __launch_bounds__(kMainThreads, 1) void k_fused_main(FusedParams p)
{
    constexpr int NT = N / 16;            // n-tiles of the state
    constexpr int PTW = 4 * NT / kWaves;  // p-tiles per wavefront in the right factor (one n-tile each)
    constexpr int KN = N / 32;            // K-steps over n
    constexpr int HBS = N + 8;            // LDS row stride of the bf16 state
    constexpr int XV = kP * kQ / 8 / kMainThreads;   // x vectors (8 bf16) per thread
    static_assert(PTW == 2 || PTW == 4, "N = 64 or 128");
    static_assert(kMainThreads >= kQ, "a thread per token of the chunk");
    static_assert(kP * HBS <= kP * kQS, "state fits in the XW region");
    __shared__ __attribute__((aligned(16))) MainSmem<N> sm;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, r = lane & 15, lg = lane >> 4;
    if (tid == 0) sm.ticket = atomicAdd(p.ticket, 1);
    __syncthreads();
    const int work = sm.ticket;
    const int nHG = static_cast<int>(p.H / p.HG);
    const int per_c = static_cast<int>(p.b) * nHG;
    const int c = work / per_c;
    const int b = (work % per_c) / nHG;
    const int hg = work % nHG;
    const int h0 = hg * static_cast<int>(p.HG);
    const int g = h0 / static_cast<int>(p.H / p.G);
    const int64_t c0 = static_cast<int64_t>(c) * kQ;
    const int L = static_cast<int>(kQ < p.T - c0 ? kQ : p.T - c0);
    const u16* xp = static_cast<const u16*>(p.x);
    const u16* Cp = static_cast<const u16*>(p.C);
    u16* yp = static_cast<u16*>(p.y);
    const int64_t PN = static_cast<int64_t>(kP) * N;
    const bool has_prev = c > 0, has_next = c + 1 < p.nC;

    // strips (16-token t-tiles) of this wavefront: balanced causal work (9 K-steps)
    int strip[2];
    strip[0] = wave;
    strip[1] = kNQ - 1 - wave;
    // state tiles of this wavefront in the right factor: n-tile ntw, p-tiles pt0..pt0+PTW-1
    const int ntw = (PTW == 4) ? wave : (wave & 3);
    const int pt0 = (PTW == 4) ? 0 : 2 * (wave >> 2);

    // ---- Gram tiles of the chunk into LDS (shared by the HG heads) -----------
    {
        const uint4* gsrc = reinterpret_cast<const uint4*>(
            p.gram + ((static_cast<int64_t>(b) * p.G + g) * p.nC + c) * kTiles * 256);
        uint4* gdst = reinterpret_cast<uint4*>(sm.GR);
        for (int i = tid; i < kTiles * 256 / 8; i += kMainThreads) gdst[i] = gsrc[i];
    }
    const u16* bt = p.BT + ((static_cast<int64_t>(b) * p.G + g) * p.nC + c) * N * kQ;
    uint4 xr[XV];
    float csr = 0.f, dtr = 0.f;
    SSD_LOAD_X(h0);
    SSD_LOAD_SCALARS(h0);
    SSD_STORE_SCALARS();
    SSD_STORE_X();
    __syncthreads();

    for (int hk = 0; hk < p.HG; ++hk) {
        const int h = h0 + hk;
        // B^T fragments of this wavefront's n-tile (L2), used after the diagonal block
        bf16x8_t btf[kQ / 32];
#pragma unroll
        for (int m = 0; m < kQ / 32; ++m)
            btf[m] = as_bf16x8(*reinterpret_cast<const uint4*>(
                bt + static_cast<int64_t>(16 * ntw + r) * kQ + 32 * m + 8 * lg));
        if (hk + 1 < p.HG) {   // prefetch the next head while this one computes
            SSD_LOAD_X(h + 1);
            SSD_LOAD_SCALARS(h + 1);
        }

        // ---- diagonal block: Y^T[p][t] for the four strips ----------------------
        f32x4_t y[2][4];
#pragma unroll
        for (int k4 = 0; k4 < 2; ++k4)
#pragma unroll
            for (int pt = 0; pt < 4; ++pt) y[k4][pt] = zero4();
#pragma unroll
        for (int k4 = 0; k4 < 2; ++k4)
            strip_diag(sm.XT, sm.cs, sm.vf, sm.dt, sm.GR, strip[k4], r, lg, lane, y[k4]);

        // ---- right factor: S[p][n], this wavefront's p-tiles x its n-tile ----------
        f32x4_t sacc[PTW];
#pragma unroll
        for (int i = 0; i < PTW; ++i) sacc[i] = zero4();
#pragma unroll
        for (int m = 0; m < kQ / 32; ++m) {
#pragma unroll
            for (int i = 0; i < PTW; ++i) {
                const bf16x8_t a = as_bf16x8(*reinterpret_cast<const uint4*>(&sm.XW[(16 * (pt0 + i) + r) * kQS + 32 * m + 8 * lg]));
                sacc[i] = mfma(a, btf[m], sacc[i]);
            }
        }

        // C fragments of the strips (L2), used by the left factor after the state exchange
        bf16x8_t cf[2][KN];
#pragma unroll
        for (int k4 = 0; k4 < 2; ++k4) {
            const int t = 16 * strip[k4] + r;
#pragma unroll
            for (int k = 0; k < KN; ++k) {
                uint4 v = make_uint4(0, 0, 0, 0);
                if (t < L) v = *reinterpret_cast<const uint4*>(Cp + ((b * p.T + c0 + t) * p.G + g) * N + 32 * k + 8 * lg);
                cf[k4][k] = as_bf16x8(v);
            }
        }

        // ---- centre factor: state entering the chunk, state leaving it ----------
        float* ring_h = p.ring + (static_cast<int64_t>(b) * p.H + h) * 2 * PN;
        const __amdgpu_buffer_rsrc_t ring_rs =
            __builtin_amdgcn_make_buffer_rsrc(ring_h, 0, static_cast<int>(2 * PN * sizeof(float)), 0x00020000);
        const int frag_base = wave * PTW * 64 + lane;   // private ring layout: [wave][frag][lane][4]
        if (has_prev && tid == 0) {
            const int* flag = p.flags + (static_cast<int64_t>(b) * p.H + h) * p.nC + (c - 1);
            long long spins = 0;
            while (__hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0) {
                __builtin_amdgcn_s_sleep(2);
                if (++spins > kSpinLimit) {
                    __hip_atomic_store(p.ticket + 1, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    break;
                }
            }
        }
        __syncthreads();   // flag seen; every wavefront is done reading XW
        f32x4_t hprev[PTW];
        if (has_prev) {
            const int slot = (c + 1) & 1;
#pragma unroll
            for (int i = 0; i < PTW; ++i) {
                const int off = static_cast<int>((slot * PN + (frag_base + i * 64) * 4) * sizeof(float));
                hprev[i] = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(ring_rs, off, 0, 16));
            }
        } else if (p.init) {
            const float* hi = p.init + (static_cast<int64_t>(b) * p.H + h) * PN;
#pragma unroll
            for (int i = 0; i < PTW; ++i)
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    hprev[i][v] = hi[(16 * (pt0 + i) + 4 * lg + v) * N + 16 * ntw + r];
        } else {
#pragma unroll
            for (int i = 0; i < PTW; ++i) hprev[i] = zero4();
        }
        const float decay = exp2f(sm.cs[kQ - 1]);
        u16* HB = sm.XW;
#pragma unroll
        for (int i = 0; i < PTW; ++i) {
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                HB[(16 * (pt0 + i) + 4 * lg + v) * HBS + 16 * ntw + r] = to_bf16(hprev[i][v]);
                sacc[i][v] = decay * hprev[i][v] + sacc[i][v];
            }
        }
        if (has_next) {
            const int slot = c & 1;
#pragma unroll
            for (int i = 0; i < PTW; ++i) {
                const int off = static_cast<int>((slot * PN + (frag_base + i * 64) * 4) * sizeof(float));
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(uint4_t, sacc[i]), ring_rs, off, 0, 16);
            }
        } else if (p.fin) {
            float* fo = p.fin + (static_cast<int64_t>(b) * p.H + h) * PN;
#pragma unroll
            for (int i = 0; i < PTW; ++i)
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    fo[(16 * (pt0 + i) + 4 * lg + v) * N + 16 * ntw + r] = sacc[i][v];
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        wait_vmem();
        __syncthreads();
        if (tid == 0 && has_next)
            __hip_atomic_store(p.flags + (static_cast<int64_t>(b) * p.H + h) * p.nC + c, 1,
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

        // ---- left factor: Y^T += exp2(cs_t) * (h_{c-1} C_t^T), strip by strip -------
#pragma unroll
        for (int k4 = 0; k4 < 2; ++k4) {
            f32x4_t tq[4];
#pragma unroll
            for (int pt = 0; pt < 4; ++pt) tq[pt] = zero4();
#pragma unroll
            for (int k = 0; k < KN; ++k) {
#pragma unroll
                for (int pt = 0; pt < 4; ++pt) {
                    const bf16x8_t aop = as_bf16x8(*reinterpret_cast<const uint4*>(&HB[(16 * pt + r) * HBS + 32 * k + 8 * lg]));
                    tq[pt] = mfma(aop, cf[k4][k], tq[pt]);
                }
            }
            const float ev = exp2f(sm.cs[16 * strip[k4] + r]);
#pragma unroll
            for (int pt = 0; pt < 4; ++pt)
#pragma unroll
                for (int v = 0; v < 4; ++v) y[k4][pt][v] += ev * tq[pt][v];
        }

        // ---- skip term and store -------------------------------------------------
        {
            const float Dh = p.D ? p.D[h] : 0.f;
#pragma unroll
            for (int k4 = 0; k4 < 2; ++k4) {
                const int t = 16 * strip[k4] + r;
                if (t < L) {
#pragma unroll
                    for (int pt = 0; pt < 4; ++pt) {
                        u16 o[4];
#pragma unroll
                        for (int v = 0; v < 4; ++v) {
                            const int pp = 16 * pt + 4 * lg + v;
                            o[v] = to_bf16(y[k4][pt][v] + Dh * bf(sm.XT[pp * kQS + t]));
                        }
                        uint2 packed;
                        packed.x = static_cast<u32>(o[0]) | (static_cast<u32>(o[1]) << 16);
                        packed.y = static_cast<u32>(o[2]) | (static_cast<u32>(o[3]) << 16);
                        *reinterpret_cast<uint2*>(yp + ((b * p.T + c0 + t) * p.H + h) * kP + 16 * pt + 4 * lg) = packed;
                    }
                }
            }
        }
        __syncthreads();   // XT, XW and the scalars are rewritten for the next head
        if (hk + 1 < p.HG) {
            SSD_STORE_SCALARS();
            SSD_STORE_X();
            __syncthreads();
        }
    }
}

template <int N>
hipError_t launch_n(const FusedParams& p, hipStream_t stream)
{
    const dim3 g_prep(static_cast<unsigned>(p.nC), static_cast<unsigned>(p.b * p.G), kPrepParts);
    hipLaunchKernelGGL(k_fused_prep<N>, g_prep, dim3(kPrepThreads), 0, stream, p);
    const unsigned nwork = static_cast<unsigned>(p.nC * p.b * (p.H / p.HG));
    hipLaunchKernelGGL(k_fused_main<N>, dim3(nwork), dim3(kMainThreads), 0, stream, p);
    return hipGetLastError();
}

}  // namespace

bool fused_supported(int64_t P, int64_t N, int64_t Q, bool bf16, bool varlen)
{
    return bf16 && !varlen && P == kP && Q == kQ && (N == 64 || N == 128);
}

FusedLayout fused_layout(int64_t b, int64_t H, int64_t N, int64_t G, int64_t nC)
{
    auto al = [](size_t v) { return (v + 255) / 256 * 256; };
    FusedLayout w;
    size_t off = 0;
    w.cs2 = off;
    off = al(off + sizeof(float) * static_cast<size_t>(b * H * nC * kQ));
    w.dtT = off;
    off = al(off + sizeof(float) * static_cast<size_t>(b * H * nC * kQ));
    w.gram = off;
    off = al(off + sizeof(u16) * static_cast<size_t>(b * G * nC) * kTiles * 256);
    w.BT = off;
    off = al(off + sizeof(u16) * static_cast<size_t>(b * G * nC) * static_cast<size_t>(N * kQ));
    w.ring = off;
    off = al(off + sizeof(float) * static_cast<size_t>(b * H) * 2 * kP * static_cast<size_t>(N));
    w.flags = off;
    off = al(off + sizeof(int) * static_cast<size_t>(b * H * nC));
    w.ticket = off;
    off = al(off + 2 * sizeof(int));
    w.total = off;
    return w;
}

hipError_t launch_fused(const FusedParams& p, hipStream_t stream)
{
    return p.N == 64 ? launch_n<64>(p, stream) : launch_n<128>(p, stream);
}

}  // namespace ssd
