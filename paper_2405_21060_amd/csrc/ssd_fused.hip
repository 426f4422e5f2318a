// Fused SSD forward for the Mamba-2 layer shapes: bf16 activations, head
// dimension P = 64, state N in {64, 128, 256} (256: two column blocks of
// 128), chunk Q = 256; plain rows, or one packed row of sequences (Section
// 8.3) through a chunk table built on the device.
//
// Two launches per call (a packed row adds the small kernels that build and
// order its chunk table).
//
// k_fused_prep, up to four workgroups per (batch, chunk, group):
//   * B^T of the chunk (N x Q, bf16), the operand layout the chunk-state
//     contraction needs (contraction over tokens);
//   * the Gram matrix C B^T of the chunk (Section 5, eq. ssm-quad: G = C B^T),
//     only its causal 16x16 tiles, stored in the exact per-lane accumulator
//     layout in which the main kernel's wavefronts hold them.
//
// k_fused_main, persistent workgroups (8 wavefronts, one per compute unit)
// taking work items (chunk, batch, group of HG heads) from a ticket counter in
// chunk-major order (a packed row's chunks by their index within their
// sequence, k_seq_order):
//   * per item: the chunk's Gram tiles (shared by the HG heads) are copied to
//     LDS asynchronously, B^T and C fragments loaded into registers; per head,
//     x (Q x P, token-major, swizzled) lands in a double-buffered LDS slot while
//     the previous head computes, and MFMA operand fragments of x^T are read
//     from it with transposing LDS reads (ds_read_b64_tr_b16);
//   * step 1: a = dt*A and its chunk-local inclusive cumsum in log2 units, one
//     token per thread, with the per-token weights of the next two steps;
//   * diagonal block (Section 6.1): Y^T = x^T (L o G)^T dt, the 1-SS mask
//     applied to the Gram fragments in registers and fed straight back into the
//     matrix cores (accumulator layout -> operand layout by permuting the
//     contraction index);
//   * right factor (Section 6.2): S = sum_s dt_s exp(cs_end - cs_s) x_s B_s^T;
//   * centre factor (Section 6.2, scalar scan of Appendix B, sequential
//     chunk-to-chunk state passing): wait for the state entering the chunk,
//     publish h_c = exp(cs_end) h_{c-1} + S for the next chunk (or write the
//     final state);
//   * left factor: Y^T += exp(cs_t) (h_{c-1} C_t^T), then + D x, rounded to
//     bf16, staged in LDS over the head's x and written as full 128-byte rows
//     with streaming stores.
//
// Cross-workgroup state passing.  States go through a two-slot ring per
// (batch, head); h_c is written with device-coherent (sc1) stores, the stores
// are drained (s_waitcnt vmcnt(0)), then a per-(batch, head, chunk) flag is
// set with a device-coherent store.  The successor polls the flag and reads
// the state with device-coherent loads.  No cache-wide writeback/invalidate is
// needed because every access to shared data is device-coherent.  Workgroups
// take their work item from a ticket counter in dispatch order, so a
// workgroup only ever waits on an item already owned by a running or finished
// workgroup; the wait is additionally bounded: when it gives up it sets the
// call's status word (which the host reads back as SSD_ERR_STATE_TIMEOUT)
// and goes on, so that every wavefront still exits.
// Two ring slots suffice: chunk c+2 overwrites the slot of chunk c only after
// reading the state of chunk c+1, which chunk c+1 published only after it had
// read (consumed) the state of chunk c.
#include <algorithm>
#include <cstdlib>
#include <utility>

#include "ssd_device.h"
#include "ssd_internal.h"

namespace ssd {
namespace {

constexpr int kQ = 256;                       // chunk length
constexpr int kNQ = kQ / 16;                  // 16-token strips per chunk
constexpr int kTiles = kNQ * (kNQ + 1) / 2;   // causal 16x16 tiles (s-tile <= t-tile)
constexpr int kP = 64;                        // head dimension
constexpr int kNH = 128;                      // widest column block of the state the chunk kernel handles at once
constexpr int kWaves = 8;
constexpr int kMainThreads = kWaves * 64;
constexpr int kPrepThreads = 512;

typedef unsigned short u16;
typedef uint32_t u32;
typedef u32 uint4_t __attribute__((ext_vector_type(4)));

struct U16x8 {
    u16 v[8];
};

__device__ __forceinline__ float bf(u16 u) { return __uint_as_float(static_cast<u32>(u) << 16); }

// Two floats -> packed bf16 pair (hardware conversion, round to nearest even).
__device__ __forceinline__ u32 pack_bf16x2(float lo, float hi)
{
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    bf16x2_t v;
    v[0] = static_cast<__bf16>(lo);
    v[1] = static_cast<__bf16>(hi);
    return __builtin_bit_cast(u32, v);
}

__device__ __forceinline__ u16 to_bf16(float f) { return static_cast<u16>(pack_bf16x2(f, 0.f)); }

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

// Inclusive prefix sum over the 64 lanes of a wavefront, in registers (DPP):
// shifts by 1, 2, 4 and 8 lanes scan each 16-lane row; broadcasts of lane 15
// (into rows 1 and 3) and of lane 31 (into rows 2 and 3) carry the row totals
// upward.  Lanes without a source add the `old` operand, zero.
__device__ __forceinline__ float wave_inclusive_scan(float v)
{
#define SSD_DPP_ADD(ctrl, rows) \
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), ctrl, rows, 0xF, false))
    SSD_DPP_ADD(0x111, 0xF);   // row_shr:1
    SSD_DPP_ADD(0x112, 0xF);   // row_shr:2
    SSD_DPP_ADD(0x114, 0xF);   // row_shr:4
    SSD_DPP_ADD(0x118, 0xF);   // row_shr:8
    SSD_DPP_ADD(0x142, 0xA);   // row_bcast:15
    SSD_DPP_ADD(0x143, 0xC);   // row_bcast:31
#undef SSD_DPP_ADD
    return v;
}

// The value of the last lane of this lane's 16-lane row.
__device__ __forceinline__ float row_last(float v, int lane)
{
    const int i = __float_as_int(v);
    const int r0 = __builtin_amdgcn_readlane(i, 15), r1 = __builtin_amdgcn_readlane(i, 31);
    const int r2 = __builtin_amdgcn_readlane(i, 47), r3 = __builtin_amdgcn_readlane(i, 63);
    const int g = lane >> 4;
    return __int_as_float(g == 0 ? r0 : g == 1 ? r1 : g == 2 ? r2 : r3);
}

// Drain this wavefront's outstanding vector-memory operations.
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Workgroup barrier for LDS data only.  __syncthreads() also waits for every
// outstanding global -> LDS copy (vmcnt(0)), which would expose the latency of
// copies issued ahead for a later head; here those copies are waited for
// explicitly (wait_vmem) where their data is first needed.  The wavefront-scope
// fences keep the compiler from moving memory accesses across the barrier;
// lgkmcnt(0) completes this wavefront's LDS accesses before it.
__device__ __forceinline__ void lds_barrier()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_s_waitcnt(0xC07F);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ float ld_coherent(const float* p)
{
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void st_coherent(float* p, float v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Column of token s in row p of the token-major LDS arrays (XT, XW): the
// 8-token group is XOR-ed with p/8 so that the transposing writes of rows
// 8 apart fall into different banks.  Groups of 4 and 8 aligned tokens stay
// contiguous.
__device__ __forceinline__ int swz(int p, int s) { return s ^ (((p >> 3) & 7) << 3); }

// B^T rows (one per state column n, Q tokens) are stored in MFMA operand
// order: within each 32-token block m, physical group g = 0..3 of 8 holds
// tokens 32m + 4g .. + 3 and then 32m + 16 + 4g .. + 3, the eight
// contraction slots one lane of a 16x16x32 MFMA operand takes (see
// load_bt_block), so that it loads them with one 16-byte load.
__device__ __forceinline__ int bt_token(int so, int e)
{
    return 32 * (so >> 2) + 4 * (so & 3) + (e < 4 ? e : 12 + e);
}

// Causal tile index of (s-tile j, t-tile i), j <= i.
__device__ __forceinline__ int tile_index(int i, int j) { return i * (i + 1) / 2 + j; }

// ---------------------------------------------------------------------------
// prep
// ---------------------------------------------------------------------------

constexpr int kGramParts = 4;   // Gram / B^T workgroups per (batch, chunk, group)

// LDS of the prep kernel: the chunk's B rows and the 64 C rows of a part's
// t-tiles (row stride N + 8 so that the 16 rows an MFMA operand reads start in
// different banks), or the dt block of the cumsum workgroups.
template <int N>
struct PrepSmem {
    u16 B[kQ * (N + 8)];
    u16 C[64 * (N + 8)];
};

// Gram workgroup (chunk c, batch b / group g, part z < 4): B rows (and the C
// rows it needs) of the chunk into LDS; the causal Gram tiles of t-tile rows
// {z, 7 - z, 8 + z, 15 - z} on MFMA (34 tiles, two wavefronts per row); a
// quarter of B^T from LDS; z == 0 also zeroes the flags of (b, c, g) and, once,
// the ticket counter.
// ---------------------------------------------------------------------------
// packed row: the chunk table (Section 8.3: sequences packed into one row, the
// state reset at every sequence start)
// ---------------------------------------------------------------------------
// First token of every sequence: where seq_idx changes (ids outside [0, nseq)
// are ignored; the caller guarantees ids 0 .. nseq-1 in order).
__global__ __launch_bounds__(256) void k_seq_starts(const int32_t* __restrict__ seq_idx, int T, int nseq,
                                                    int* __restrict__ starts)
{
    const int t = blockIdx.x * 256 + threadIdx.x;
    if (t == 0) starts[nseq] = T;
    if (t >= T) return;
    const int v = seq_idx[t];
    if ((t == 0 || seq_idx[t - 1] != v) && v >= 0 && v < nseq) starts[v] = t;
}

// The same from starts given by value (host offsets).
__global__ __launch_bounds__(256) void k_seq_starts_args(SeqStartsArg a, int* __restrict__ starts)
{
    for (int i = threadIdx.x; i <= a.n; i += 256) starts[i] = a.v[i];
}

constexpr int kTabThreads = 1024;

// Exclusive prefix sum over the workgroup (kTabThreads lanes), plus the total.
__device__ long long block_exclusive_sum(long long v, long long* s_w, long long* total)
{
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    long long inc = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const long long u = __shfl_up(inc, d);
        if (lane >= d) inc += u;
    }
    if (lane == 63) s_w[w] = inc;
    __syncthreads();
    long long before = 0, all = 0;
    for (int k = 0; k < kTabThreads / 64; ++k) {
        before += k < w ? s_w[k] : 0;
        all += s_w[k];
    }
    __syncthreads();   // s_w is reused by the next call
    *total = all;
    return before + inc - v;
}

// The chunks of every sequence, in token order (one workgroup): sequence r
// of length len gives ceil(len / Q) chunks from its first token on.  Every
// entry stays inside [0, T) and the table's capacity whatever the ids hold.
// seq_first (may be null): the table index of each sequence's first chunk,
// then the number of entries.
template <int Q>
__global__ __launch_bounds__(kTabThreads) void k_seq_chunks(const int* __restrict__ starts, int T, int nseq,
                                                            int cap, int ring_cap, int4* __restrict__ vtab,
                                                            int* __restrict__ seq_first, int* __restrict__ vcount)
{
    __shared__ long long s_w[kTabThreads / 64];
    // 64-bit sums: ids that break the contract may describe more chunks than T
    long long base = 0, rbase = 0;
    for (int r0 = 0; r0 < nseq; r0 += kTabThreads) {
        const int r = r0 + static_cast<int>(threadIdx.x);
        int st = 0, len = 0;
        if (r < nseq) {
            st = min(max(starts[r], 0), T);
            len = min(max(starts[r + 1], st), T) - st;
        }
        const int nch = len / Q + (len % Q != 0 ? 1 : 0);
        long long tot = 0, rtot = 0;
        const long long v0 = base + block_exclusive_sum(nch, s_w, &tot);
        const long long rr = rbase + block_exclusive_sum(nch > 1 ? 1 : 0, s_w, &rtot);
        const int ring = static_cast<int>(rr < ring_cap ? rr : ring_cap - 1);
        for (int k = 0; k < nch && v0 + k < cap; ++k) {
            const int flags = (k == 0 ? 1 : 0) | (k == nch - 1 ? 2 : 0) | (ring << 2);
            vtab[v0 + k] = make_int4(st + k * Q, min(Q, len - k * Q), r, flags);
        }
        if (seq_first && r < nseq) seq_first[r] = static_cast<int>(v0 < cap ? v0 : cap);
        base += tot;
        rbase += rtot;
    }
    if (threadIdx.x == 0) {
        *vcount = static_cast<int>(base < cap ? base : cap);
        if (seq_first) seq_first[nseq] = *vcount;
    }
}

// The order in which the chunk kernel takes a packed row's table entries:
// by the entry's index within its sequence (every sequence's first chunk,
// then every second chunk, ...; one workgroup).  In table order the items
// taken together are consecutive chunks of one or two sequences, each
// waiting for the one before it; in this order they are mostly of different
// sequences, and a chunk's predecessor was taken about a round earlier.  Any
// order that puts a chunk after the chunk before it in its sequence keeps the
// chunk kernel deadlock-free, and the order of the entries of one index
// (here the order of LDS atomics) changes no result.  Rows of more than
// kOrderDepths chunks keep the table order.
constexpr int kOrderDepths = 8192;

template <int Q>
__global__ __launch_bounds__(kTabThreads) void k_seq_order(const int4* __restrict__ vtab,
                                                           const int* __restrict__ starts,
                                                           const int* __restrict__ vcount, int T,
                                                           int* __restrict__ vorder)
{
    __shared__ int pos[kOrderDepths];
    __shared__ long long s_w[kTabThreads / 64];
    const int n = *vcount;
    const int depths = T / Q + (T % Q != 0 ? 1 : 0);   // no sequence has more chunks
    if (depths > kOrderDepths) {
        for (int e = threadIdx.x; e < n; e += kTabThreads) vorder[e] = e;
        return;
    }
    // index of entry e within its sequence: its first token's distance from the
    // sequence's first token (clamped as the table kernel clamps it), in chunks
    const auto depth = [&](int e) {
        const int4 v = vtab[e];
        const int st = min(max(starts[v.z], 0), T);
        return min(max((v.x - st) / Q, 0), depths - 1);
    };
    for (int k = threadIdx.x; k < depths; k += kTabThreads) pos[k] = 0;
    __syncthreads();
    for (int e = threadIdx.x; e < n; e += kTabThreads) atomicAdd(&pos[depth(e)], 1);
    __syncthreads();
    // entries per index -> first position of each index
    long long base = 0;
    for (int k0 = 0; k0 < depths; k0 += kTabThreads) {
        const int k = k0 + static_cast<int>(threadIdx.x);
        long long tot = 0;
        const long long first = base + block_exclusive_sum(k < depths ? pos[k] : 0, s_w, &tot);
        if (k < depths) pos[k] = static_cast<int>(first);   // only this thread reads pos[k] in this pass
        base += tot;
    }
    __syncthreads();
    for (int e = threadIdx.x; e < n; e += kTabThreads) vorder[atomicAdd(&pos[depth(e)], 1)] = e;
}

// PACKED: a packed row, chunk positions from the chunk table.
template <int N, bool PACKED>
__global__ __launch_bounds__(kPrepThreads) void k_fused_prep(FusedParams p)
{
    constexpr int RS = N + 8;
    __shared__ __attribute__((aligned(16))) PrepSmem<(N > kNH ? kNH : N)> sm;
    const int c = blockIdx.x;
    const int b = static_cast<int>(blockIdx.y / p.G), g = static_cast<int>(blockIdx.y % p.G);
    const int tid = threadIdx.x, lane = tid & 63, r = lane & 15, lg = lane >> 4;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int hpg = static_cast<int>(p.H / p.G);
    if (blockIdx.z == 0 && blockIdx.x == 0 && blockIdx.y == 0 && tid == 0) {
        p.ticket[0] = 0;
        if (p.reset_status) *p.status = 0;   // set by the chunk kernel when a state wait gives up
    }
    int64_t c0 = static_cast<int64_t>(c) * kQ;
    int L = static_cast<int>(kQ < p.T - c0 ? kQ : p.T - c0);
    if constexpr (PACKED) {   // packed row: chunk c of the table (entries past its end: nothing to do)
        if (c >= *p.vcount) return;
        const int4 e = p.vtab[c];
        c0 = e.x;
        L = e.y;
    }

    if constexpr (N > kNH) {
        // The state's width (N = 256) is wider than LDS holds B for: the Gram
        // contraction runs in passes over column blocks of B and C (NP
        // columns each), the tiles accumulating in registers.
        constexpr int NP = kNH, RSP = NP + 8;
        const int64_t brow = p.G * N;
        const u16* Bchunk = static_cast<const u16*>(p.B) + ((b * p.T + c0) * p.G + g) * N;
        const u16* Cchunk = static_cast<const u16*>(p.C) + ((b * p.T + c0) * p.G + g) * N;
        u16* gram = p.gram + ((static_cast<int64_t>(b) * p.G + g) * p.nC + c) * kTiles * 256;
        u16* bt = p.BT + ((static_cast<int64_t>(b) * p.G + g) * p.nC + c) * N * kQ;
        for (int part = blockIdx.z; part < kGramParts; part += gridDim.z) {
            if (part != static_cast<int>(blockIdx.z)) __syncthreads();   // the previous part's LDS reads are done
            if (part == 0)
                for (int hh = tid; hh < hpg; hh += kPrepThreads)
                    p.flags[(static_cast<int64_t>(b) * p.H + g * hpg + hh) * p.nC + c] = 0;
            const int rows[4] = {part, 7 - part, 8 + part, kNQ - 1 - part};
            const int i = rows[wave >> 1];   // this wavefront's t-tile row; s-tiles (wave & 1) + 2 k
            f32x4_t acc[kNQ / 2];
#pragma unroll
            for (int k = 0; k < kNQ / 2; ++k) acc[k] = zero4();
#pragma unroll 1
            for (int kp = 0; kp < N / NP; ++kp) {
                if (kp > 0) __syncthreads();   // the previous block's LDS reads are done
                constexpr int kBPer = kQ * NP / 8 / kPrepThreads, kCPer = 64 * NP / 8 / kPrepThreads;
                static_assert(kBPer * kPrepThreads == kQ * NP / 8 && kCPer * kPrepThreads == 64 * NP / 8, "split");
                uint4 vb[kBPer], vc[kCPer];
#pragma unroll
                for (int k = 0; k < kBPer; ++k) {
                    const int e = tid + kPrepThreads * k;
                    const int s = e / (NP / 8), col = 8 * (e % (NP / 8));
                    vb[k] = *reinterpret_cast<const uint4*>(Bchunk + (s < L ? s : L - 1) * brow + kp * NP + col);
                }
#pragma unroll
                for (int k = 0; k < kCPer; ++k) {
                    const int e = tid + kPrepThreads * k;
                    const int lr = e / (NP / 8), col = 8 * (e % (NP / 8));
                    const int t = 16 * rows[lr >> 4] + (lr & 15);
                    vc[k] = *reinterpret_cast<const uint4*>(Cchunk + (t < L ? t : L - 1) * brow + kp * NP + col);
                }
#pragma unroll
                for (int k = 0; k < kBPer; ++k) {
                    const int e = tid + kPrepThreads * k;
                    const int s = e / (NP / 8), col = 8 * (e % (NP / 8));
                    *reinterpret_cast<uint4*>(&sm.B[s * RSP + col]) = (s < L) ? vb[k] : make_uint4(0, 0, 0, 0);
                }
#pragma unroll
                for (int k = 0; k < kCPer; ++k) {
                    const int e = tid + kPrepThreads * k;
                    const int lr = e / (NP / 8), col = 8 * (e % (NP / 8));
                    const int t = 16 * rows[lr >> 4] + (lr & 15);
                    *reinterpret_cast<uint4*>(&sm.C[lr * RSP + col]) = (t < L) ? vc[k] : make_uint4(0, 0, 0, 0);
                }
                __syncthreads();
                uint4 cfr[NP / 32];
#pragma unroll
                for (int k = 0; k < NP / 32; ++k)
                    cfr[k] = *reinterpret_cast<const uint4*>(&sm.C[(16 * (wave >> 1) + r) * RSP + 32 * k + 8 * lg]);
#pragma unroll
                for (int kk = 0; kk < kNQ / 2; ++kk) {
                    const int j = (wave & 1) + 2 * kk;
                    if (j <= i)
#pragma unroll
                        for (int k = 0; k < NP / 32; ++k) {
                            const uint4 va =
                                *reinterpret_cast<const uint4*>(&sm.B[(16 * j + r) * RSP + 32 * k + 8 * lg]);
                            acc[kk] = mfma(as_bf16x8(va), as_bf16x8(cfr[k]), acc[kk]);
                        }
                }
                // this part's quarter of this block's B^T rows: item (n, 8 tokens), 16-byte stores along s
                constexpr int kBtItems = NP * (kQ / 8) / kGramParts;
                for (int e = part * kBtItems + tid; e < (part + 1) * kBtItems; e += kPrepThreads) {
                    const int n = e % NP, so = e / NP;
                    U16x8 v;
#pragma unroll
                    for (int q8 = 0; q8 < 8; ++q8) v.v[q8] = sm.B[bt_token(so, q8) * RSP + n];
                    *reinterpret_cast<uint4*>(bt + static_cast<int64_t>(kp * NP + n) * kQ + 8 * so) =
                        __builtin_bit_cast(uint4, v);
                }
            }
#pragma unroll
            for (int kk = 0; kk < kNQ / 2; ++kk) {
                const int j = (wave & 1) + 2 * kk;
                if (j <= i) {
                    uint2 packed;
                    packed.x = pack_bf16x2(acc[kk][0], acc[kk][1]);
                    packed.y = pack_bf16x2(acc[kk][2], acc[kk][3]);
                    *reinterpret_cast<uint2*>(gram + (static_cast<int64_t>(tile_index(i, j)) * 64 + lane) * 4) = packed;
                }
            }
        }
    } else {
    // A workgroup takes parts z, z + gridDim.z, ... of the chunk (fewer
    // workgroups per chunk when there are many chunks: the B rows stay in LDS).
    for (int part = blockIdx.z; part < kGramParts; part += gridDim.z) {
        const bool first = part == static_cast<int>(blockIdx.z);
        if (!first) __syncthreads();   // the previous part's LDS reads are done
        // ---- flags of this (batch, chunk) and group
        if (part == 0)
            for (int hh = tid; hh < hpg; hh += kPrepThreads)
                p.flags[(static_cast<int64_t>(b) * p.H + g * hpg + hh) * p.nC + c] = 0;
        // t-tile rows of this part (balanced: 34 tiles)
        const int rows[4] = {part, 7 - part, 8 + part, kNQ - 1 - part};

        // ---- B rows of the chunk and C rows of this part's t-tiles into LDS (rows
        // past a partial chunk: zeros).  C row tile rows[k] lands at LDS row 16 k.
        const u16* Bchunk = static_cast<const u16*>(p.B) + ((b * p.T + c0) * p.G + g) * N;
        const u16* Cchunk = static_cast<const u16*>(p.C) + ((b * p.T + c0) * p.G + g) * N;
        const int64_t brow = p.G * N;
        // all loads are issued before any LDS store, so that they are in flight together
        constexpr int kBPer = kQ * N / 8 / kPrepThreads, kCPer = 64 * N / 8 / kPrepThreads;
        static_assert(kBPer * kPrepThreads == kQ * N / 8 && kCPer * kPrepThreads == 64 * N / 8, "even split");
        uint4 vb[kBPer], vc[kCPer];
        if (first)
#pragma unroll
        for (int k = 0; k < kBPer; ++k) {
            const int i = tid + kPrepThreads * k;
            const int s = i / (N / 8), col = 8 * (i % (N / 8));
            vb[k] = *reinterpret_cast<const uint4*>(Bchunk + (s < L ? s : L - 1) * brow + col);
        }
#pragma unroll
        for (int k = 0; k < kCPer; ++k) {
            const int i = tid + kPrepThreads * k;
            const int lr = i / (N / 8), col = 8 * (i % (N / 8));
            const int t = 16 * rows[lr >> 4] + (lr & 15);
            vc[k] = *reinterpret_cast<const uint4*>(Cchunk + (t < L ? t : L - 1) * brow + col);
        }
        if (first)
#pragma unroll
        for (int k = 0; k < kBPer; ++k) {
            const int i = tid + kPrepThreads * k;
            const int s = i / (N / 8), col = 8 * (i % (N / 8));
            *reinterpret_cast<uint4*>(&sm.B[s * RS + col]) = (s < L) ? vb[k] : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int k = 0; k < kCPer; ++k) {
            const int i = tid + kPrepThreads * k;
            const int lr = i / (N / 8), col = 8 * (i % (N / 8));
            const int t = 16 * rows[lr >> 4] + (lr & 15);
            *reinterpret_cast<uint4*>(&sm.C[lr * RS + col]) = (t < L) ? vc[k] : make_uint4(0, 0, 0, 0);
        }
        __syncthreads();

        // ---- Gram tiles G^T[s][t] = sum_n B_s[n] C_t[n] (bf16), accumulator layout per lane.
        // Wavefront w: row rows[w / 2], s-tiles j = w%2, w%2 + 2, ...
        u16* gram = p.gram + ((static_cast<int64_t>(b) * p.G + g) * p.nC + c) * kTiles * 256;
        {
            const int i = rows[wave >> 1];
            uint4 cfr[N / 32];
#pragma unroll
            for (int k = 0; k < N / 32; ++k)
                cfr[k] = *reinterpret_cast<const uint4*>(&sm.C[(16 * (wave >> 1) + r) * RS + 32 * k + 8 * lg]);
#pragma unroll 1
            for (int j = wave & 1; j <= i; j += 2) {
                f32x4_t acc = zero4();
#pragma unroll
                for (int k = 0; k < N / 32; ++k) {
                    const uint4 va = *reinterpret_cast<const uint4*>(&sm.B[(16 * j + r) * RS + 32 * k + 8 * lg]);
                    acc = mfma(as_bf16x8(va), as_bf16x8(cfr[k]), acc);
                }
                uint2 packed;
                packed.x = pack_bf16x2(acc[0], acc[1]);
                packed.y = pack_bf16x2(acc[2], acc[3]);
                *reinterpret_cast<uint2*>(gram + (static_cast<int64_t>(tile_index(i, j)) * 64 + lane) * 4) = packed;
            }
        }

        // ---- this part's quarter of B^T from LDS: item (n, 8 tokens), 16-byte stores along s
        u16* bt = p.BT + ((static_cast<int64_t>(b) * p.G + g) * p.nC + c) * N * kQ;
        constexpr int kBtItems = N * (kQ / 8) / kGramParts;
        for (int i = part * kBtItems + tid; i < (part + 1) * kBtItems; i += kPrepThreads) {
            const int n = i % N, so = i / N;
            U16x8 v;
#pragma unroll
            for (int e = 0; e < 8; ++e) v.v[e] = sm.B[bt_token(so, e) * RS + n];
            *reinterpret_cast<uint4*>(bt + static_cast<int64_t>(n) * kQ + 8 * so) = __builtin_bit_cast(uint4, v);
        }
    }
    }
}

// ---------------------------------------------------------------------------
// main
// ---------------------------------------------------------------------------
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
typedef __attribute__((address_space(3))) void lds_void;

// x of one head lives token-major in LDS: row s = 64 features (128 bytes),
// its eight 16-byte groups XOR-swizzled by (s & 7) so that the transposing
// reads of 4 consecutive rows spread over the banks.
__device__ __forceinline__ int xs_off(int s, int p) { return s * kP + ((((p >> 3) ^ (s & 7)) << 3) | (p & 7)); }

// ds_read_b64_tr_b16 within each 16-lane group: source lane j reads row
// k0 + j/4, features f0 + 4 (j%4) .. +3; lane i then holds feature f0 + i of
// rows k0 .. k0+3 -- an MFMA operand fragment (4 contraction slots) of x^T.
__device__ __forceinline__ uint2 xfrag(const u16* xs, int k0, int f0, int lane)
{
    const int j = lane & 15;
    const u16* a = xs + xs_off(k0 + (j >> 2), f0 + 4 * (j & 3));
    return __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(a)));
}

// LDS of the chunk kernel.  The Gram tiles and the bf16 state are separate
// __shared__ objects (declared in the kernel) so that the compiler can tell
// that copies into them never alias the reads of this struct's buffers.
template <int N>
struct MainSmem {
    u16 XS[2][kQ * kP];       // x of the current / next head (token-major, swizzled)
    float cs[2][kQ];          // chunk-local cumsum of dt A (log2 units) of the current / next head
    float dt[2][kQ];
    float wtot[2][4];         // per-wavefront totals of the cumsum
    float wn[kP];             // normalisation weights of the current head
    float vf[2][kQ];          // dt_s exp2(cs[tile end] - cs_s)
    float w[2][kQ];           // dt_s exp2(cs[Q-1] - cs_s)
    int ticket;
};

// Transposing read at a precomputed LDS byte address (see x_tr_base).
__device__ __forceinline__ uint2 tr_read(const char* a)
{
    return __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(a)));
}

// Byte offset, within a head's x buffer, of this lane's transposing read of
// rows 4 lg + (lane%16)/4 (+ 32 m, + 16), features f0 + 4 (lane%4) .. +3.
// Adding a multiple of 8 to the row leaves the swizzle unchanged, so the reads
// of every K-step m and of the upper half (+16 rows) are this offset plus the
// constants 4096 m and 2048.
__device__ __forceinline__ int x_tr_base(int f0, int lane)
{
    const int j = lane & 15, lg = lane >> 4;
    return 2 * xs_off(4 * lg + (j >> 2), f0 + 4 * (j & 3));
}

__device__ __forceinline__ void unpack4(uint2 gp, float* g)
{
    g[0] = __uint_as_float(gp.x << 16);
    g[1] = __uint_as_float(gp.x & 0xFFFF0000u);
    g[2] = __uint_as_float(gp.y << 16);
    g[3] = __uint_as_float(gp.y & 0xFFFF0000u);
}

// Off-diagonal s-tile (entirely before the strip): the 1-SS mask factors as
// exp2(cs_t - cs_end(j)) * exp2(cs_end(j) - cs_s), both factors <= 1, the
// second folded with dt_s into vf.
__device__ __forceinline__ void mask_off(uint2 gp, float u, float4 vf4, float* mv)
{
    float g[4];
    unpack4(gp, g);
    mv[0] = g[0] * (u * vf4.x);
    mv[1] = g[1] * (u * vf4.y);
    mv[2] = g[2] * (u * vf4.z);
    mv[3] = g[3] * (u * vf4.w);
}

// The strip's own s-tile: exp2(cs_t - cs_s) dt_s directly for s <= t, zero
// above the diagonal (branch-free: exponent clamped, upper triangle selected away).
__device__ __forceinline__ void mask_diag(uint2 gp, int t, int sb, float cst, float4 cs4, float4 dt4,
                                          float* mv)
{
    float g[4];
    unpack4(gp, g);
    const float csv[4] = {cs4.x, cs4.y, cs4.z, cs4.w}, dtv[4] = {dt4.x, dt4.y, dt4.z, dt4.w};
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        const float e = __builtin_amdgcn_exp2f(fminf(cst - csv[v], 0.f));
        mv[v] = (sb + v <= t) ? g[v] * (e * dtv[v]) : 0.f;
    }
}

// One K-step (s-tiles 2m, 2m+1) of strip S: masked Gram operand, 4 MFMAs.
template <int S, int M>
__device__ __forceinline__ void strip_step(const uint4* af, const char* gbase, int t, float cst,
                                           float ce0, float ce1, float4 vf0, float4 vf1,
                                           const float* cs, const float* dt, int lg, f32x4_t* yv)
{
    constexpr int j0 = 2 * M, j1 = 2 * M + 1;
    float mv[8];
    const uint2 g0 = *reinterpret_cast<const uint2*>(gbase + j0 * 512);
    if constexpr (j1 < S) {
        const uint2 g1 = *reinterpret_cast<const uint2*>(gbase + j1 * 512);
        mask_off(g0, __builtin_amdgcn_exp2f(cst - ce0), vf0, mv);
        mask_off(g1, __builtin_amdgcn_exp2f(cst - ce1), vf1, mv + 4);
    } else if constexpr (j1 == S) {
        const uint2 g1 = *reinterpret_cast<const uint2*>(gbase + j1 * 512);
        const int sb1 = 16 * j1 + 4 * lg;
        mask_off(g0, __builtin_amdgcn_exp2f(cst - ce0), vf0, mv);
        mask_diag(g1, t, sb1, cst, *reinterpret_cast<const float4*>(cs + sb1),
                  *reinterpret_cast<const float4*>(dt + sb1), mv + 4);
    } else {   // j0 == S
        const int sb0 = 16 * j0 + 4 * lg;
        mask_diag(g0, t, sb0, cst, *reinterpret_cast<const float4*>(cs + sb0),
                  *reinterpret_cast<const float4*>(dt + sb0), mv);
#pragma unroll
        for (int v = 4; v < 8; ++v) mv[v] = 0.f;
    }
    const bf16x8_t bop = pack8(mv);
#pragma unroll
    for (int pt = 0; pt < 4; ++pt) yv[pt] = mfma(as_bf16x8(af[pt]), bop, yv[pt]);
}

// One K-step m of the right factor S[p][n] += sum_s x[s][p] w_s B[s][n] for this
// wavefront's p-tiles PT0 .. PT0 + PTW - 1 (its n-tile's B^T fragment bt, scaled
// by w here), from x^T fragments already in registers.
template <int PTW, int PT0>
__device__ __forceinline__ void rf_step(const uint4* af, uint4 bt, const float* wl, int m, f32x4_t* sacc)
{
    const float4 w0 = *reinterpret_cast<const float4*>(wl + 32 * m);
    const float4 w1 = *reinterpret_cast<const float4*>(wl + 32 * m + 16);
    const float wv[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
    const u32 bw[4] = {bt.x, bt.y, bt.z, bt.w};
    float bf8[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        bf8[2 * e] = __uint_as_float(bw[e] << 16) * wv[2 * e];
        bf8[2 * e + 1] = __uint_as_float(bw[e] & 0xFFFF0000u) * wv[2 * e + 1];
    }
    const bf16x8_t bop = pack8(bf8);
#pragma unroll
    for (int i = 0; i < PTW; ++i) sacc[i] = mfma(as_bf16x8(af[PT0 + i]), bop, sacc[i]);
}

// Diagonal block of wavefront W, whose strips (t-tiles) are W and 15 - W
// (9 K-steps between them for every W).  K-step m covers s-tiles 2m, 2m+1; its
// contraction index is permuted to the Gram accumulator layout (slot e<4 ->
// s = 32m + 4 lg + e, e>=4 -> s = 32m + 16 + 4 lg + e - 4), and the x^T
// fragments and vf of a K-step are read once for both strips.  Everything
// about the strips is a compile-time constant, so the body is straight-line
// code with immediate LDS offsets.
// PTW > 0: the right factor (this wavefront's n-tile, PTW p-tiles) runs in the
// same pass, on the x^T fragments the diagonal block has read (its first nB
// K-steps; the rest read their own), so that x is read from LDS once for both.
// `mid` runs after K-step kMidStep, `fin` once the Gram rows have been read for
// the last time.
constexpr int kMidStep = 0;   // K-step after which `mid` runs (the next head's x copy)
template <int W, int PTW, class Mid, class Fin>
__device__ __forceinline__ void diag_wave(const char* xsb, const int* xa, const float* cs,
                                          const float* vf, const float* dt, const float* wrf, const uint4* btf,
                                          const u16* GR, int r, int lg, int lane, f32x4_t* yA, f32x4_t* yB,
                                          f32x4_t* sacc, const Mid& mid, const Fin& fin)
{
    constexpr int sA = W, sB = 15 - W;
    constexpr int nA = sA / 2 + 1, nB = sB / 2 + 1;
    const int tA = 16 * sA + r, tB = 16 * sB + r;
    const float csA = cs[tA], csB = cs[tB];
    const char* gA = reinterpret_cast<const char*>(GR) + tile_index(sA, 0) * 512 + 8 * lane;
    const char* gB = reinterpret_cast<const char*>(GR) + tile_index(sB, 0) * 512 + 8 * lane;
    const float* vfl = vf + 4 * lg;
    const char* x0 = xsb + xa[0];
    const char* x1 = xsb + xa[1];
    const char* x2 = xsb + xa[2];
    const char* x3 = xsb + xa[3];
    constexpr int kPt0 = PTW == 4 ? 0 : 2 * (W >> 2);   // the right factor's first p-tile
    const float* wrl = wrf + 4 * lg;
    // Software pipeline: the LDS operands of K-step m+1 are requested before
    // the masking and MFMAs of K-step m.
    struct Step {
        uint4 af[4];
        float4 vf0, vf1;
        float ce0, ce1;
    };
    auto load = [&](int m, Step& d) {
        const uint2 l0 = tr_read(x0 + 4096 * m), h0 = tr_read(x0 + 4096 * m + 2048);
        const uint2 l1 = tr_read(x1 + 4096 * m), h1 = tr_read(x1 + 4096 * m + 2048);
        const uint2 l2 = tr_read(x2 + 4096 * m), h2 = tr_read(x2 + 4096 * m + 2048);
        const uint2 l3 = tr_read(x3 + 4096 * m), h3 = tr_read(x3 + 4096 * m + 2048);
        d.af[0] = make_uint4(l0.x, l0.y, h0.x, h0.y);
        d.af[1] = make_uint4(l1.x, l1.y, h1.x, h1.y);
        d.af[2] = make_uint4(l2.x, l2.y, h2.x, h2.y);
        d.af[3] = make_uint4(l3.x, l3.y, h3.x, h3.y);
        d.vf0 = *reinterpret_cast<const float4*>(vfl + 32 * m);
        d.vf1 = *reinterpret_cast<const float4*>(vfl + 32 * m + 16);
        d.ce0 = cs[32 * m + 15];
        d.ce1 = cs[32 * m + 31];
    };
    Step cur;
    load(0, cur);
    [&]<int... Ms>(std::integer_sequence<int, Ms...>) {
        ([&] {
            constexpr int m = Ms;
            Step nxt;
            if constexpr (m + 1 < nB) load(m + 1, nxt);
            strip_step<sB, m>(cur.af, gB, tB, csB, cur.ce0, cur.ce1, cur.vf0, cur.vf1, cs, dt, lg, yB);
            if constexpr (m < nA)
                strip_step<sA, m>(cur.af, gA, tA, csA, cur.ce0, cur.ce1, cur.vf0, cur.vf1, cs, dt, lg, yA);
            if constexpr (m + 1 == nB) fin();   // this wavefront's Gram rows are read for the last time
            if constexpr (PTW > 0) rf_step<PTW, kPt0>(cur.af, btf[m], wrl, m, sacc);
            if constexpr (m == kMidStep) mid();
            if constexpr (m + 1 < nB) cur = nxt;
        }(), ...);
    }(std::make_integer_sequence<int, nB>{});
    if constexpr (PTW > 0) {
        // the right factor's remaining K-steps
        const char* xp[4] = {x0, x1, x2, x3};
        [&]<int... Ms>(std::integer_sequence<int, Ms...>) {
            ([&] {
                constexpr int m = nB + Ms;
                uint4 af[4];
#pragma unroll
                for (int i = 0; i < PTW; ++i) {
                    const uint2 lo = tr_read(xp[kPt0 + i] + 4096 * m), hi = tr_read(xp[kPt0 + i] + 4096 * m + 2048);
                    af[kPt0 + i] = make_uint4(lo.x, lo.y, hi.x, hi.y);
                }
                rf_step<PTW, kPt0>(af, btf[m], wrl, m, sacc);
                if constexpr (m == kMidStep) mid();
            }(), ...);
        }(std::make_integer_sequence<int, kQ / 32 - nB>{});
    }
}

template <int PTW, class Mid, class Fin>
__device__ __forceinline__ void diag_block(int wave, const char* xsb, const int* xa, const float* cs,
                                           const float* vf, const float* dt, const float* wrf, const uint4* btf,
                                           const u16* GR, int r, int lg, int lane, f32x4_t* yA, f32x4_t* yB,
                                           f32x4_t* sacc, const Mid& mid, const Fin& fin)
{
#define SSD_DIAG_WAVE(W) diag_wave<W, PTW>(xsb, xa, cs, vf, dt, wrf, btf, GR, r, lg, lane, yA, yB, sacc, mid, fin)
    switch (wave) {
    case 0: SSD_DIAG_WAVE(0); break;
    case 1: SSD_DIAG_WAVE(1); break;
    case 2: SSD_DIAG_WAVE(2); break;
    case 3: SSD_DIAG_WAVE(3); break;
    case 4: SSD_DIAG_WAVE(4); break;
    case 5: SSD_DIAG_WAVE(5); break;
    case 6: SSD_DIAG_WAVE(6); break;
    default: SSD_DIAG_WAVE(7); break;
    }
#undef SSD_DIAG_WAVE
}

// One work item of the chunk kernel: (chunk, batch row, group of HG heads).
struct Item {
    int c, b, h0, g, L;
    int seq, ring;       // row of the initial / final states, row of the state ring
    int64_t c0;
    int64_t rows;        // tokens readable from c0 on (the rest of the row or sequence)
    const u16* xchunk;   // x at token c0, head 0
    const u16* cchunk;   // C at token c0, group g
    bool has_prev, has_next;
};

template <bool PACKED>
__device__ __forceinline__ Item decode_item(const FusedParams& p, int work, int per_c, int nHG, int N)
{
    Item it;
    it.c = work / per_c;
    if constexpr (PACKED)
        if (p.vorder) it.c = p.vorder[it.c];   // the table entry taken in this place
    it.b = (work % per_c) / nHG;
    it.h0 = (work % nHG) * static_cast<int>(p.HG);
    it.g = it.h0 / static_cast<int>(p.H / p.G);
    if constexpr (PACKED) {   // packed row (batch 1): chunk it.c of the sequence chunk table
        const int4 e = p.vtab[it.c];
        it.c0 = e.x;
        it.L = e.y;
        it.rows = e.y;
        it.seq = e.z;
        it.ring = e.w >> 2;
        it.has_prev = (e.w & 1) == 0;
        it.has_next = (e.w & 2) == 0;
    } else {
        it.c0 = static_cast<int64_t>(it.c) * kQ;
        it.L = static_cast<int>(kQ < p.T - it.c0 ? kQ : p.T - it.c0);
        it.rows = p.T - it.c0;
        it.seq = it.b;
        it.ring = it.b;
        it.has_prev = it.c > 0;
        it.has_next = it.c + 1 < p.nC;
    }
    it.xchunk = static_cast<const u16*>(p.x) + (static_cast<int64_t>(it.b) * p.T + it.c0) * p.H * kP;
    it.cchunk = static_cast<const u16*>(p.C) + ((static_cast<int64_t>(it.b) * p.T + it.c0) * p.G + it.g) * N;
    return it;
}

// Asynchronous global -> LDS copies (buffer_load ... lds, 16 bytes per lane,
// landing at the LDS address in M0 + 16 lane).  They are issued through inline
// assembly so that the compiler, which cannot tell which LDS bytes such a copy
// writes, does not make every later LDS access wait for it; every read of
// copied data is preceded by an explicit wait (s_waitcnt vmcnt) and a barrier.
// A copy adds to the vector-memory counter like any load, so the compiler's
// own waits for its loads stay correct (they can only wait longer).
typedef int i32x4 __attribute__((ext_vector_type(4)));

// Buffer descriptor (raw, no stride) over `bytes` bytes from `base`; reads past
// the end return zeros.  The base is uniform across the wavefront.
__device__ __forceinline__ i32x4 buffer_rsrc(const void* base, int64_t bytes)
{
    const unsigned long long a = reinterpret_cast<unsigned long long>(base);
    i32x4 r;
    r[0] = __builtin_amdgcn_readfirstlane(static_cast<int>(a & 0xFFFFFFFFull));
    r[1] = __builtin_amdgcn_readfirstlane(static_cast<int>((a >> 32) & 0xFFFFull));
    r[2] = __builtin_amdgcn_readfirstlane(static_cast<int>(bytes < 0x7FFFFFFF ? bytes : 0x7FFFFFFF));
    r[3] = 0x00020000;
    return r;
}

__device__ __forceinline__ void copy16_to_lds(i32x4 rsrc, const void* lds_dst, int voffset, int soffset)
{
    const unsigned m0 =
        __builtin_amdgcn_readfirstlane(static_cast<unsigned>(reinterpret_cast<uintptr_t>(lds_dst)));
    asm volatile("buffer_load_dwordx4 %0, %1, %2 offen lds"
                 :: "v"(voffset), "s"(rsrc), "s"(soffset), "{m0}"(m0) : "memory");
}

// Per-lane byte offsets of the copies, fixed for the whole kernel.
struct DmaOffsets {
    int x[4];   // x: token row s = 8 (4 wave + i) + lane/8, physical 16-byte group lane%8
    int l16;    // 16 lane
};

__device__ __forceinline__ DmaOffsets dma_offsets(const FusedParams& p, int wave, int lane)
{
    DmaOffsets o;
    const int xrow_bytes = static_cast<int>(p.H * kP * 2);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int s = 8 * (4 * wave + i) + (lane >> 3);
        const int grp = (lane & 7) ^ (s & 7);   // logical group stored at physical slot lane%8
        o.x[i] = s * xrow_bytes + 16 * grp;
    }
    o.l16 = 16 * lane;
    return o;
}

// Copy of head hh's x (an item's chunk) into the LDS buffer xdst: 4 blocks of
// 8 tokens per wavefront (lane l of a block fetches the 16 bytes that land at
// block + 16 l).  The descriptor ends at the end of the batch row, so rows
// past a partial last chunk read as zeros (such tokens have dt = 0 and zero
// Gram rows and columns, and are never stored).
__device__ __forceinline__ void dma_head(const FusedParams& p, const Item& it, int hh, u16* xdst, int wave,
                                         const DmaOffsets& o)
{
    const i32x4 xrs = buffer_rsrc(it.xchunk, it.rows * p.H * kP * 2);
    const int hoff = hh * kP * 2;
#pragma unroll
    for (int i = 0; i < 4; ++i) copy16_to_lds(xrs, xdst + (4 * wave + i) * 512, o.x[i], hoff);
}

// Copy of head hh's gate branch z, rows of the two strips of this wavefront,
// into the LDS buffer zdst with x's swizzled layout: 4 blocks of 8 rows (lane
// l of a block fetches the 16 bytes that land at block + 16 l).  Rows past a
// partial last chunk read as zeros (they are never stored).
__device__ __forceinline__ void dma_z_strips(const FusedParams& p, const Item& it, int hh, u16* zdst,
                                             const int* strip, int lane)
{
    const u16* zchunk = static_cast<const u16*>(p.z) + (static_cast<int64_t>(it.b) * p.T + it.c0) * p.H * kP;
    const i32x4 zrs = buffer_rsrc(zchunk, it.rows * p.H * kP * 2);
    const int row_bytes = static_cast<int>(p.H * kP * 2);
#pragma unroll
    for (int k4 = 0; k4 < 2; ++k4)
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int s0 = 16 * strip[k4] + 8 * i;   // first row of the block
            const int s = s0 + (lane >> 3);
            const int grp = (lane & 7) ^ (s & 7);    // logical group landing at physical slot lane % 8
            copy16_to_lds(zrs, zdst + s0 * kP, s * row_bytes + 16 * grp, hh * kP * 2);
        }
}

// dt of token `tid` (clamped to the chunk) of head hh of an item, raw bf16.
__device__ __forceinline__ u16 load_dt(const FusedParams& p, const Item& it, int hh, int tid)
{
    const int t = tid < it.L ? tid : it.L - 1;
    return static_cast<const u16*>(p.dt)[(it.b * p.T + it.c0 + t) * p.H + hh];
}

// The chunk's causal Gram tiles (shared by the item's heads) into LDS.
__device__ __forceinline__ void dma_gram(u16* gr, const FusedParams& p, const Item& it, int wave,
                                         const DmaOffsets& o)
{
    constexpr int kBlocks = kTiles * 256 * 2 / 1024;
    const i32x4 rs = buffer_rsrc(p.gram + ((static_cast<int64_t>(it.b) * p.G + it.g) * p.nC + it.c) * kTiles * 256,
                                 kBlocks * 1024);
    for (int blk = wave; blk < kBlocks; blk += kWaves) copy16_to_lds(rs, gr + blk * 512, o.l16, blk * 1024);
}

// The Gram tile rows {wave, 15 - wave} of an item (the only rows this
// wavefront's diagonal block reads) into LDS: 1 KiB copies, the last one of
// the odd-length row by half the lanes -- 9 copies for every wavefront.
__device__ __forceinline__ void dma_gram_rows(u16* gr, const FusedParams& p, const Item& it, int wave, int lane)
{
    const i32x4 rs = buffer_rsrc(p.gram + ((static_cast<int64_t>(it.b) * p.G + it.g) * p.nC + it.c) * kTiles * 256,
                                 kTiles * 512);
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int row = k == 0 ? wave : kNQ - 1 - wave;
        const int off = tile_index(row, 0) * 512, bytes = (row + 1) * 512;
        for (int o = 0; o < bytes; o += 1024)
            if (bytes - o >= 1024 || lane < 32) copy16_to_lds(rs, gr + (off + o) / 2, 16 * lane, off + o);
    }
}

// B^T fragments of n-tile ntw of column block hf (NH columns) of the state
// for the right factor, in the diagonal block's contraction order (slots 0-3:
// tokens 32m + 4 lg + e, slots 4-7: 32m + 16 + 4 lg + e - 4), so that both
// share the x^T reads.
template <int N, int NH>
__device__ __forceinline__ void load_bt_block(const FusedParams& p, const Item& it, int ntw, int r, int lg, int hf,
                                              uint4 (&btf)[kQ / 32])
{
    const u16* bt = p.BT + ((static_cast<int64_t>(it.b) * p.G + it.g) * p.nC + it.c) * N * kQ;
    const u16* btr = bt + (static_cast<unsigned>(hf * NH + 16 * ntw + r) * kQ + 8u * lg);
#pragma unroll
    for (int m = 0; m < kQ / 32; ++m) btf[m] = *reinterpret_cast<const uint4*>(btr + 32 * m);
}

// The item-level B^T fragments: the first column block of the state (the
// only one for N <= 128; with two, every head loads the second block's own).
template <int N>
__device__ __forceinline__ void load_bt(const FusedParams& p, const Item& it, int ntw, int r, int lg,
                                        uint4 (&btf)[kQ / 32])
{
    load_bt_block<N, (N < kNH ? N : kNH)>(p, it, ntw, r, lg, 0, btf);
}

// C fragments of the two strips for the left factor, columns [hf NH, hf NH +
// NH) of C (rows past a partial chunk's end are clamped; they are never stored).
template <int N, int NH>
__device__ __forceinline__ void load_c_block(const FusedParams& p, const Item& it, const int* strip, int r, int lg,
                                             int hf, uint4 (&cf)[2][NH / 32])
{
    const unsigned crow = static_cast<unsigned>(p.G * N);
#pragma unroll
    for (int k4 = 0; k4 < 2; ++k4) {
        const int t = 16 * strip[k4] + r;
        const unsigned tc = static_cast<unsigned>(t < it.L ? t : it.L - 1);
#pragma unroll
        for (int k = 0; k < NH / 32; ++k)
            cf[k4][k] = *reinterpret_cast<const uint4*>(it.cchunk + (tc * crow + hf * NH + 32u * k + 8u * lg));
    }
}

// One head of a work item.  Every LDS buffer is a separate __restrict__
// parameter: the compiler then knows that the asynchronous copies into the
// next head's buffers (and the next item's Gram tiles) never alias the buffers
// read here, and does not make those reads wait for the copies.
// Y32: y is written in float32 straight from the accumulators (the layer
// recomputed for the block gradients, whose dy and dz need y before rounding).
// FUSE: the right factor (of the first column block of the state, with two)
// runs in the diagonal block's pass over x.
template <int N, bool PACKED, bool EARLY, bool Y32, bool FUSE>
__device__ __forceinline__ void head_step(const FusedParams& p, const Item& it, int hk, int& next, int nwork,
                                          int per_c, int nHG,
                                          uint4 (&btf)[kQ / 32], uint4 (&cf)[2][(N < kNH ? N : kNH) / 32],
                                          u16& dtr, bool& ready, u16* __restrict__ xs, u16* __restrict__ xs_n,
                                          float* __restrict__ cs, float* __restrict__ dt,
                                          float* __restrict__ wt, float* __restrict__ vf, float* __restrict__ w,
                                          float* __restrict__ cs_n, float* __restrict__ dt_n,
                                          float* __restrict__ wt_n, float* __restrict__ vf_n, float* __restrict__ w_n,
                                          u16* __restrict__ gr, u16* __restrict__ hb, int* __restrict__ tk,
                                          const float* __restrict__ A_logp, const float* __restrict__ Dp,
                                          const float* __restrict__ biasp, float* __restrict__ wn)
{
    // The state (P x N) is processed in HALVES column blocks of NH <= 128
    // (two for N = 256): right factor, state passing and left factor each
    // per block, so that registers and the LDS copy of the state stay those of
    // N = 128.
    constexpr int NH = N < kNH ? N : kNH;
    constexpr int HALVES = N / NH;
    constexpr int NT = NH / 16;
    constexpr int PTW = 4 * NT / kWaves;
    constexpr int KN = NH / 32;
    constexpr int HBS = NH + 8;
    // per-wavefront constants (loop-invariant; the compiler keeps them out of the loops)
    const int tid = threadIdx.x, lane = tid & 63, r = lane & 15, lg = lane >> 4;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // provably uniform
    // strips (16-token t-tiles) of this wavefront: balanced causal work (9 K-steps)
    const int strip[2] = {wave, kNQ - 1 - wave};
    // state tiles of this wavefront in the right factor: n-tile ntw, p-tiles pt0..pt0+PTW-1
    const int ntw = (PTW == 4) ? wave : (wave & 3);
    const int pt0 = (PTW == 4) ? 0 : 2 * (wave >> 2);
    int xa[4];   // byte offsets of this lane's transposing x reads, per p-tile
#pragma unroll
    for (int pt = 0; pt < 4; ++pt) xa[pt] = x_tr_base(16 * pt, lane);
    const DmaOffsets dmo = dma_offsets(p, wave, lane);
    u16* yp = static_cast<u16*>(p.y);
    const int64_t PN = static_cast<int64_t>(kP) * N;
    const unsigned xrow = static_cast<unsigned>(p.H * kP);

    const int h = it.h0 + hk;
    const bool last = hk + 1 == p.HG;
    const int b = it.b, c = it.c, L = it.L;
    const int64_t c0 = it.c0;
    const bool has_prev = it.has_prev, has_next = it.has_next;
    const float Dh = Dp ? Dp[h] : 0.f;   // scalar loads (read-only kernel arguments)
    // this head's normalisation weights (one per thread of the first wavefront),
    // stored to LDS at the state barrier, read by the output stage
    const bool gate = p.z != nullptr, norm = p.norm_head != 0;
    float wreg = 0.f;
    if (norm && tid < kP) wreg = p.norm_weight ? p.norm_weight[h * kP + tid] : 1.f;
    // x (and this thread's dt) of the next head -- of this item, or of the next
    // item once known -- arrive while this head computes
    u16 dtr_next = 0;
    int h_next = -1, L_next = 0;   // the next head of this workgroup, once known
    if (!last) {
        if (tid < kQ) dtr_next = load_dt(p, it, h + 1, tid);
        h_next = h + 1;
        L_next = L;
    } else if (hk > 0 && next < nwork) {
        const Item nit = decode_item<PACKED>(p, next, per_c, nHG, N);
        if (tid < kQ) dtr_next = load_dt(p, nit, nit.h0, tid);
        h_next = nit.h0;
        L_next = nit.L;
    }

    // Two column blocks of the state: the first block's B^T fragments are the
    // item's (btf, shared by its heads); the second block's are this head's own,
    // requested when the first block's right factor starts.
    uint4 bth[kQ / 32];

    // ---- step 1: chunk-local inclusive cumsum of a = dt A (log2 units), one token
    // per thread (wavefront scans, then the wavefront totals through LDS), and the
    // per-token weights of the diagonal block and the right factor.  The head
    // before this one in the workgroup has normally done it already, in its
    // output stage (`ready`); otherwise (a workgroup's first head) here.
    // The scan for head hh of a chunk of Lh tokens: this thread's dt, its
    // wavefront prefix, the wavefront totals to wtv.
    const auto scan = [&](u16 raw, int hh, int Lh, float* wtv, float& dv, float& inc) {
        dv = 0.f;
        inc = 0.f;
        if (tid < kQ) {
            if (tid < Lh) {
                dv = bf(raw);
                if (p.dtx.active) {   // the block path's dt parameterisation
                    if (biasp) dv += biasp[hh];
                    if (p.dtx.softplus) dv = softplus_f(dv);
                    dv = fminf(fmaxf(dv, p.dtx.lo), p.dtx.hi);
                }
            }
            inc = dv * (-expf(A_logp[hh]) * kLog2e);
            inc = wave_inclusive_scan(inc);
            if (lane == 63) wtv[wave] = inc;
        }
    };
    // ... and, after a barrier, the cumsum and the weights
    const auto weights = [&](const float* wtv, float dv, float inc, float* csv, float* dtv, float* vfv, float* wv) {
        if (tid < kQ) {
            float pre = 0.f, tot = 0.f;
#pragma unroll
            for (int k = 0; k < kQ / 64; ++k) {
                const float v = wtv[k];
                tot += v;
                if (k < wave) pre += v;
            }
            const float cst = inc + pre;
            const float cend = row_last(cst, lane);   // end of this token's 16-token tile
            csv[tid] = cst;
            dtv[tid] = dv;
            vfv[tid] = dv * exp2f(cend - cst);
            wv[tid] = dv * exp2f(tot - cst);
        }
    };
    if (!ready) {
        float d, incl;
        scan(dtr, h, L, wt, d, incl);
        lds_barrier();
        weights(wt, d, incl, cs, dt, vf, w);
        lds_barrier();
    }

    // ---- diagonal block: Y^T[p][t] for the two strips ------------------------
    // (with one column block of the state, the right factor S[p][n] = sum_s
    // x[s][p] w_s B[s][n] of this wavefront's tiles runs in the same pass: x is
    // read from LDS once for both)
    f32x4_t y[2][4];
#pragma unroll
    for (int k4 = 0; k4 < 2; ++k4)
#pragma unroll
        for (int pt = 0; pt < 4; ++pt) y[k4][pt] = zero4();
    f32x4_t sacc[HALVES][PTW];
#pragma unroll
    for (int hf = 0; hf < HALVES; ++hf)
#pragma unroll
        for (int i = 0; i < PTW; ++i) sacc[hf][i] = zero4();
    // Opaque to the optimiser, so that it does not hoist the unpacking of B^T out
    // of the head loop (64 more registers, and a wait for the loads at the start
    // of every item).
    const auto opaque_bt = [&] {
#pragma unroll
        for (int m = 0; m < kQ / 32; ++m) {
            uint4_t v = __builtin_bit_cast(uint4_t, btf[m]);
            asm volatile("" : "+v"(v));
            btf[m] = __builtin_bit_cast(uint4, v);
        }
    };
    // x of the next head -- of this item, or of the next item once known --
    // arrives while this head computes.  It is requested after the diagonal
    // block's first K-step (FUSE) or after the diagonal block, not at the head's
    // start, where the copies queue behind the previous head's y stores; not
    // much later either, since the state passing's own loads wait for it (the
    // wait is in issue order).
    const auto next_x = [&] {
        if (!last)
            dma_head(p, it, h + 1, xs_n, wave, dmo);
        else if (hk > 0 && next < nwork) {
            const Item nit = decode_item<PACKED>(p, next, per_c, nHG, N);
            dma_head(p, nit, nit.h0, xs_n, wave, dmo);
        }
    };
    // Last head of an item with the next item known: each wavefront refills the
    // Gram rows of its own two strips for the next item (no other wavefront
    // reads them), well ahead of that item's diagonal block: right after its
    // diagonal block, or -- in the fused pass with N >= 128 -- as soon as the
    // block has read them for the last time, before the right factor's
    // remaining K-steps (2.7B layer 0.1878 -> 0.1856 ms; with N = 64, and
    // outside the fused pass, that placement measured 0.5-2 % slower).
    constexpr bool kGramInPass = FUSE && N >= kNH;
    constexpr bool kBtInPass = FUSE && N == kNH;
    const bool gram_early = last && hk > 0 && next < nwork;
    const auto gram_refill = [&] {
        if (gram_early) dma_gram_rows(gr, p, decode_item<PACKED>(p, next, per_c, nHG, N), wave, lane);
    };
    const auto gram_fin = [&] {
        if constexpr (kGramInPass) gram_refill();
    };
    if constexpr (FUSE) {
        opaque_bt();
        diag_block<PTW>(wave, reinterpret_cast<const char*>(xs), xa, cs, vf, dt, w, btf, gr, r, lg, lane, y[0], y[1],
                        sacc[0], next_x, gram_fin);
        // (two column blocks: the first block's right factor was fused; the
        // second block's B^T fragments now -- requested during the diagonal
        // block they would hold registers it needs)
        if constexpr (HALVES > 1) load_bt_block<N, NH>(p, it, ntw, r, lg, 1, bth);
    } else {
        diag_block<0>(wave, reinterpret_cast<const char*>(xs), xa, cs, vf, dt, w, btf, gr, r, lg, lane, y[0], y[1],
                      sacc[0], [] {}, [] {});
    }
    if constexpr (!kGramInPass) gram_refill();
    if constexpr (!FUSE) next_x();
    // The next item's B^T fragments, in an item's last head with the next item
    // known: with the fused right factor and N = 128 as soon as the pass has used
    // this item's (2.7B layer 0.1863 -> 0.1829 ms; with N = 64 it measured 1.6 %
    // slower, so there, as everywhere else, they follow the y stores below).
    if (kBtInPass && last && hk > 0 && next < nwork)
        load_bt<N>(p, decode_item<PACKED>(p, next, per_c, nHG, N), ntw, r, lg, btf);
    // skip term D x, while x is in LDS (with the gate branch, its buffer takes z
    // after the right factor)
#pragma unroll
    for (int k4 = 0; k4 < 2; ++k4) {
        const int t = 16 * strip[k4] + r;
#pragma unroll
        for (int pt = 0; pt < 4; ++pt) {
            const uint2 xv = *reinterpret_cast<const uint2*>(xs + xs_off(t, 16 * pt + 4 * lg));
            const float xf[4] = {__uint_as_float(xv.x << 16), __uint_as_float(xv.x & 0xFFFF0000u),
                                 __uint_as_float(xv.y << 16), __uint_as_float(xv.y & 0xFFFF0000u)};
#pragma unroll
            for (int v = 0; v < 4; ++v) y[k4][pt][v] += Dh * xf[v];
        }
    }

    // ---- right factor (of the blocks not fused above): S[p][n] = sum_s x[s][p]
    // w_s B[s][n], this wavefront's tiles, per column block of the state
    if constexpr (!FUSE) opaque_bt();
#pragma unroll
    for (int hf = FUSE ? 1 : 0; hf < HALVES; ++hf) {
        if (HALVES > 1) __builtin_amdgcn_sched_barrier(0);
        if (!FUSE && HALVES > 1 && hf + 1 < HALVES) load_bt_block<N, NH>(p, it, ntw, r, lg, hf + 1, bth);
        const uint4 (&bsrc)[kQ / 32] = hf > 0 ? bth : btf;
        const char* xsb = reinterpret_cast<const char*>(xs);
        const float* wl = w + 4 * lg;
#pragma unroll
        for (int m = 0; m < kQ / 32; ++m) {
            const float4 w0 = *reinterpret_cast<const float4*>(wl + 32 * m);
            const float4 w1 = *reinterpret_cast<const float4*>(wl + 32 * m + 16);
            const float wv[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
            const u32 bw[4] = {bsrc[m].x, bsrc[m].y, bsrc[m].z, bsrc[m].w};
            float bf8[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                bf8[2 * e] = __uint_as_float(bw[e] << 16) * wv[2 * e];
                bf8[2 * e + 1] = __uint_as_float(bw[e] & 0xFFFF0000u) * wv[2 * e + 1];
            }
            const bf16x8_t bop = pack8(bf8);
#pragma unroll
            for (int i = 0; i < PTW; ++i) {
                const char* xb = xsb + xa[pt0 + i] + 4096 * m;
                const uint2 lo = tr_read(xb), hi = tr_read(xb + 2048);
                sacc[hf][i] = mfma(as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y)), bop, sacc[hf][i]);
            }
        }
    }


    // ---- centre factor: state entering the chunk, state leaving it ----------
    float* ring_h = p.ring + (static_cast<int64_t>(it.ring) * p.H + h) * 2 * PN;
    const __amdgpu_buffer_rsrc_t ring_rs =
        __builtin_amdgcn_make_buffer_rsrc(ring_h, 0, static_cast<int>(2 * PN * sizeof(float)), 0x00020000);
    // private ring layout: [column block][wave][frag][lane][4]
    const int frag_base = wave * PTW * 64 + lane;
    // The first head reserves the next work item here: the wait for the atomic's
    // result merges with the state wait below, and the result is shared through
    // LDS at the state barrier.
    if (hk == 0 && tid == 0) *tk = atomicAdd(p.ticket, 1);
    if (has_prev && tid == 0) {
        const int* flag = p.flags + (static_cast<int64_t>(b) * p.H + h) * p.nC + (c - 1);
        long long spins = 0;
        while (__hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0) {
            if (++spins >= p.spin_limit) {   // give up: report it, never hang
                __hip_atomic_store(p.status, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                break;
            }
            __builtin_amdgcn_s_sleep(2);
        }
    }
    lds_barrier();   // flag seen by tid 0
    // The gate branch z of this head's output rows into this head's x buffer:
    // every wavefront is past the right factor, the last reader of x.  Each
    // wavefront copies the 32 rows of its own two strips, so its own wait
    // (in the output stage) suffices.
    if (gate) dma_z_strips(p, it, h, xs, strip, lane);
    const float decay = exp2f(cs[kQ - 1]);
    // this lane's first element in the caller's (P, N) initial / final state
    const int st_lo = ((16 * pt0 + 4 * lg) * N + 16 * ntw + r) * static_cast<int>(sizeof(float));
    bool gram_ahead = false;
    f32x4_t tq[2][4];
#pragma unroll
    for (int k4 = 0; k4 < 2; ++k4)
#pragma unroll
        for (int pt = 0; pt < 4; ++pt) tq[k4][pt] = zero4();
#pragma unroll
    for (int hf = 0; hf < HALVES; ++hf) {
        // (the compiler keeps each block's loads in their block: hoisting the
        // second block's would hold both blocks' operands in registers at once)
        if (HALVES > 1) __builtin_amdgcn_sched_barrier(0);
        if (hf > 0) lds_barrier();   // the previous block's left factor is done with the LDS state
        const int hoff = hf * (PN / HALVES);   // this block's offset in a ring slot (floats)
        const int coff = hf * NH * static_cast<int>(sizeof(float));   // ... and in a (P, N) state row (bytes)
        f32x4_t hprev[PTW];
        if (has_prev) {
            const int slot = (c + 1) & 1;
#pragma unroll
            for (int i = 0; i < PTW; ++i) {
                const int off = static_cast<int>((slot * PN + hoff + (frag_base + i * 64) * 4) * sizeof(float));
                hprev[i] = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(ring_rs, off, 0, 16));
            }
        } else if (p.init) {
            // (P, N) layout of the caller's initial state: lane offset + uniform row offsets
            const __amdgpu_buffer_rsrc_t irs = __builtin_amdgcn_make_buffer_rsrc(
                const_cast<float*>(p.init + (static_cast<int64_t>(it.seq) * p.H + h) * PN), 0,
                static_cast<int>(PN * sizeof(float)), 0x00020000);
#pragma unroll
            for (int i = 0; i < PTW; ++i)
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    hprev[i][v] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                        irs, st_lo + coff, (16 * i + v) * N * static_cast<int>(sizeof(float)), 0));
        } else {
#pragma unroll
            for (int i = 0; i < PTW; ++i) hprev[i] = zero4();
        }
#pragma unroll
        for (int i = 0; i < PTW; ++i) {
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                hb[(16 * (pt0 + i) + 4 * lg + v) * HBS + 16 * ntw + r] = to_bf16(hprev[i][v]);
                sacc[hf][i][v] = decay * hprev[i][v] + sacc[hf][i][v];
            }
        }
        if (has_next) {
            const int slot = c & 1;
#pragma unroll
            for (int i = 0; i < PTW; ++i) {
                const int off = static_cast<int>((slot * PN + hoff + (frag_base + i * 64) * 4) * sizeof(float));
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(uint4_t, sacc[hf][i]), ring_rs, off, 0, 16);
            }
        } else if (p.fin) {
            const __amdgpu_buffer_rsrc_t frs = __builtin_amdgcn_make_buffer_rsrc(
                p.fin + (static_cast<int64_t>(it.seq) * p.H + h) * PN, 0,
                static_cast<int>(PN * sizeof(float)), 0x00020000);
#pragma unroll
            for (int i = 0; i < PTW; ++i)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    // extract the element first: bit-casting a vector element in place is
                    // mis-lowered (component 0 stored for every v)
                    const float val = sacc[hf][i][v];
                    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(val), frs, st_lo + coff,
                                                          (16 * i + v) * N * static_cast<int>(sizeof(float)), 0);
                }
        }
        // The state stores drain while the left factor runs; the flag is set after
        // the epilogue's barrier, once every wavefront has waited for its stores.
        // Where the chain of chunks is what bounds the launch (early_flag), every
        // wavefront waits for its stores here instead and the flag follows this
        // barrier, so the next chunk need not wait for this one's left factor.
        // (EARLY: a template parameter, so that the other launches carry none of it.)
        if (hf + 1 == HALVES) {
            if (norm && tid < kP) wn[tid] = wreg;
            if constexpr (EARLY) wait_vmem();
        }
        // Two column blocks: this block's C fragments.
        uint4 cfh[2][KN];
        if constexpr (HALVES > 1) load_c_block<N, NH>(p, it, strip, r, lg, hf, cfh);
        lds_barrier();   // bf16 state (block) in LDS complete; every wavefront is past the diagonal block
        if (hf + 1 == HALVES && EARLY && tid == 0 && has_next)
            __hip_atomic_store(p.flags + (static_cast<int64_t>(b) * p.H + h) * p.nC + c, 1,
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (hf == 0) {
            if (hk == 0) next = *tk;
            // The next item's Gram tiles (and, with one head per item, its first head's
            // x): only the bf16 state and z are read from here on.
            // (With one head per item the next item is known only here: its Gram tiles
            // and its first head's x follow now, by all wavefronts.)
            gram_ahead = last && hk == 0 && next < nwork;
            if (gram_ahead) {
                const Item nit = decode_item<PACKED>(p, next, per_c, nHG, N);
                dma_gram(gr, p, nit, wave, dmo);
                dma_head(p, nit, nit.h0, xs_n, wave, dmo);
                if (tid < kQ) dtr_next = load_dt(p, nit, nit.h0, tid);
            }
        }

        // ---- left factor: Y^T += exp2(cs_t) * (h_{c-1} C_t^T) for both strips (this block's columns)
#pragma unroll
        for (int k = 0; k < KN; ++k) {
#pragma unroll
            for (int pt = 0; pt < 4; ++pt) {
                const bf16x8_t aop = as_bf16x8(*reinterpret_cast<const uint4*>(&hb[(16 * pt + r) * HBS + 32 * k + 8 * lg]));
                const uint4 c0v = HALVES > 1 ? cfh[0][k] : cf[0][k], c1v = HALVES > 1 ? cfh[1][k] : cf[1][k];
                tq[0][pt] = mfma(aop, as_bf16x8(c0v), tq[0][pt]);
                tq[1][pt] = mfma(aop, as_bf16x8(c1v), tq[1][pt]);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    }
#pragma unroll
    for (int k4 = 0; k4 < 2; ++k4) {
        const float ev = exp2f(cs[16 * strip[k4] + r]);
#pragma unroll
        for (int pt = 0; pt < 4; ++pt)
#pragma unroll
            for (int v = 0; v < 4; ++v) y[k4][pt][v] += ev * tq[k4][pt][v];
    }


    // ---- the block's gate and per-head normalisation; y staged in place over
    // this head's x (or z) buffer, then full-row stores
    {
        u16* xw = xs;
        // state stores complete (and the next head's x and this head's z have
        // landed; z was copied before the Gram tiles); the Gram copies (at most 9
        // per wavefront, at least 8) may stay in flight
        if (gram_ahead)
            __builtin_amdgcn_s_waitcnt(0x0F78);   // vmcnt(8)
        else
            wait_vmem();
        if (gate) {   // y * SiLU(z), SiLU(z) = z / (1 + 2^(-z log2 e))
#pragma unroll
            for (int k4 = 0; k4 < 2; ++k4)
#pragma unroll
                for (int pt = 0; pt < 4; ++pt) {
                    const uint2 zv = *reinterpret_cast<const uint2*>(xw + xs_off(16 * strip[k4] + r, 16 * pt + 4 * lg));
                    const float zf[4] = {__uint_as_float(zv.x << 16), __uint_as_float(zv.x & 0xFFFF0000u),
                                         __uint_as_float(zv.y << 16), __uint_as_float(zv.y & 0xFFFF0000u)};
#pragma unroll
                    for (int v = 0; v < 4; ++v)
                        y[k4][pt][v] *= zf[v] * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(-zf[v] * kLog2e));
                }
        }
        if (norm) {   // RMS over the head's P channels of each token: the four lanes r, r+16, r+32, r+48
#pragma unroll
            for (int k4 = 0; k4 < 2; ++k4) {
                float ss = 0.f;
#pragma unroll
                for (int pt = 0; pt < 4; ++pt)
#pragma unroll
                    for (int v = 0; v < 4; ++v) ss += y[k4][pt][v] * y[k4][pt][v];
                ss += __shfl_xor(ss, 16, 64);
                ss += __shfl_xor(ss, 32, 64);
                const float scale = 1.f / sqrtf(ss * (1.f / kP) + p.norm_eps);
#pragma unroll
                for (int pt = 0; pt < 4; ++pt) {
                    const float4 w4 = *reinterpret_cast<const float4*>(wn + 16 * pt + 4 * lg);
                    const float wv[4] = {w4.x, w4.y, w4.z, w4.w};
#pragma unroll
                    for (int v = 0; v < 4; ++v) y[k4][pt][v] *= scale * wv[v];
                }
            }
        }
        // step 1 of this workgroup's next head, while this head's y is written
        if (last && hk == 0 && next < nwork) {   // one head per item: known since the state barrier
            const Item nit = decode_item<PACKED>(p, next, per_c, nHG, N);
            h_next = nit.h0;
            L_next = nit.L;
        }
        float d_next = 0.f, incl_next = 0.f;
        if (h_next >= 0) scan(dtr_next, h_next, L_next, wt_n, d_next, incl_next);
        if constexpr (Y32) {
            // float32 y straight from the accumulators: lane = token 16 strip + r,
            // features 16 pt + 4 lg .. + 3 (16 bytes)
            float* y32 = static_cast<float*>(p.y) + ((static_cast<int64_t>(b) * p.T + c0) * p.H + h) * kP;
#pragma unroll
            for (int k4 = 0; k4 < 2; ++k4) {
                const int t = 16 * strip[k4] + r;
                if (t < L)
#pragma unroll
                    for (int pt = 0; pt < 4; ++pt)
                        *reinterpret_cast<float4*>(y32 + static_cast<unsigned>(t) * xrow + 16 * pt + 4 * lg) =
                            make_float4(y[k4][pt][0], y[k4][pt][1], y[k4][pt][2], y[k4][pt][3]);
            }
            lds_barrier();   // (the next head's wavefront totals)
            if (!EARLY && tid == 0 && has_next)
                __hip_atomic_store(p.flags + (static_cast<int64_t>(b) * p.H + h) * p.nC + c, 1,
                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (h_next >= 0) weights(wt_n, d_next, incl_next, cs_n, dt_n, vf_n, w_n);
            if (gram_ahead) wait_vmem();   // the next item's Gram tiles have landed
        } else {
#pragma unroll
            for (int k4 = 0; k4 < 2; ++k4) {
                const int t = 16 * strip[k4] + r;
#pragma unroll
                for (int pt = 0; pt < 4; ++pt) {
                    uint2 packed;
                    packed.x = pack_bf16x2(y[k4][pt][0], y[k4][pt][1]);
                    packed.y = pack_bf16x2(y[k4][pt][2], y[k4][pt][3]);
                    *reinterpret_cast<uint2*>(xw + xs_off(t, 16 * pt + 4 * lg)) = packed;   // cells this lane read
                }
            }
            lds_barrier();   // (y staged; the next head's wavefront totals)
            if (!EARLY && tid == 0 && has_next)
                __hip_atomic_store(p.flags + (static_cast<int64_t>(b) * p.H + h) * p.nC + c, 1,
                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (h_next >= 0) weights(wt_n, d_next, incl_next, cs_n, dt_n, vf_n, w_n);
            u16* ychunk = yp + ((static_cast<int64_t>(b) * p.T + c0) * p.H + h) * kP;
            constexpr int kPieces = kQ * kP / 8 / kMainThreads;   // 16-byte pieces per thread
            uint4 v[kPieces];
#pragma unroll
            for (int k = 0; k < kPieces; ++k) {
                const int ci = tid + kMainThreads * k;      // piece: token ci/8, group ci%8
                v[k] = *reinterpret_cast<const uint4*>(xw + xs_off(ci >> 3, 8 * (ci & 7)));
            }
            if (gram_ahead) wait_vmem();   // the next item's Gram tiles have landed
#pragma unroll
            for (int k = 0; k < kPieces; ++k) {
                const int ci = tid + kMainThreads * k;
                const int t = ci >> 3, grp = ci & 7;
                // streaming (non-temporal) stores: y is not read again by this kernel
                if (t < L) __builtin_nontemporal_store(__builtin_bit_cast(uint4_t, v[k]), reinterpret_cast<uint4_t*>(ychunk + (static_cast<unsigned>(t) * xrow + 8u * grp)));
            }
        }
    }
    // The next item's B^T fragments (their last use in this item is behind
    // us), requested after the waits above so that none of those waits for them.
    if (last && next < nwork) {
        const Item nit = decode_item<PACKED>(p, next, per_c, nHG, N);
        if (!(kBtInPass && hk > 0)) load_bt<N>(p, nit, ntw, r, lg, btf);
        if constexpr (HALVES == 1) load_c_block<N, NH>(p, nit, strip, r, lg, 0, cf);
    }
    lds_barrier();   // this head's LDS buffers may be refilled from here on; the next head's weights are in place
    dtr = dtr_next;  // here, where the load has long completed (the epilogue waited for it)
    ready = h_next >= 0;
}

// A_log, D and the dt bias come as separate read-only arguments so that their per-head values
// are scalar loads (a vector load would wait behind the outstanding copies).
template <int N, bool PACKED, bool EARLY, bool Y32, bool FUSE>
__global__ __launch_bounds__(kMainThreads, 1) void k_fused_main(FusedParams p, const float* __restrict__ A_logp,
                                                                const float* __restrict__ Dp,
                                                                const float* __restrict__ biasp)
{
    constexpr int NH = N < kNH ? N : kNH; // columns of the state per block (two blocks for N = 256)
    constexpr int NT = NH / 16;           // n-tiles of a block
    constexpr int PTW = 4 * NT / kWaves;  // p-tiles per wavefront in the right factor (one n-tile each)
    constexpr int KN = NH / 32;           // K-steps over a block's columns
    constexpr int HBS = NH + 8;           // LDS row stride of the bf16 state (one block)
    static_assert(PTW == 2 || PTW == 4, "N = 64, 128 or 256");
    static_assert(kMainThreads >= kQ && kP == 64 && kQ * kP * 2 == 32 * 1024 * 1, "x buffer = 32 KiB");
    static_assert(kQ * kP / 512 == 4 * kWaves, "x DMA: 4 blocks of 8 tokens per wavefront");
    static_assert((kTiles * 256 * 2) % 1024 == 0, "Gram DMA in 1 KiB blocks");
    __shared__ __attribute__((aligned(16))) MainSmem<N> sm;
    __shared__ __attribute__((aligned(16))) u16 s_gr[kTiles * 256];   // Gram tiles: [tile][lane][4] bf16
    __shared__ __attribute__((aligned(16))) u16 s_hb[kP * HBS];       // bf16 state entering the chunk (P x N)

    const int tid = threadIdx.x, lane = tid & 63, r = lane & 15, lg = lane >> 4;
    // wavefront index, provably uniform (branches on it stay scalar)
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int nHG = static_cast<int>(p.H / p.HG);
    const int per_c = static_cast<int>(p.b) * nHG;
    const int nwork = (PACKED ? *p.vcount : static_cast<int>(p.nC)) * per_c;
    const DmaOffsets dmo = dma_offsets(p, wave, lane);
    const int ntw = (PTW == 4) ? wave : (wave & 3);
    const int strip[2] = {wave, kNQ - 1 - wave};

    // Persistent workgroups: work items are taken from a ticket counter in
    // chunk-major order, so an item only ever waits for an item already taken
    // by a running (or finished) workgroup.  The operands of the next item are
    // prefetched during the last head of the current one.
    u16 dtr = 0;    // this thread's dt of the current head (token tid), raw bf16
    bool ready = false;   // the current head's step 1 done by the head before it
    if (tid == 0) sm.ticket = atomicAdd(p.ticket, 1);
    __syncthreads();
    int work = sm.ticket;
    if (work >= nwork) return;
    {
        const Item it = decode_item<PACKED>(p, work, per_c, nHG, N);
        dma_gram(s_gr, p, it, wave, dmo);
        dma_head(p, it, it.h0, sm.XS[0], wave, dmo);
        if (tid < kQ) dtr = load_dt(p, it, it.h0, tid);
    }
    wait_vmem();
    __syncthreads();

    int q = 0;      // LDS buffer of the current head
    // register operands shared by an item's heads (see load_bt / load_c): loaded
    // here for the first item, and for every later item by the last head of the
    // item before it, right after their last use there
    uint4 btf[kQ / 32];   // (one column block of the state; with two, each head loads its own)
    uint4 cf[2][KN];      // C fragments of the left factor (one column block; with two, per head and block)
    {
        const Item it = decode_item<PACKED>(p, work, per_c, nHG, N);
        load_bt<N>(p, it, ntw, r, lg, btf);
        if constexpr (N <= kNH) load_c_block<N, N>(p, it, strip, r, lg, 0, cf);
    }
    for (;;) {
    const Item it = decode_item<PACKED>(p, work, per_c, nHG, N);
    int next = nwork;
    for (int hk = 0; hk < p.HG; ++hk) {
        head_step<N, PACKED, EARLY, Y32, FUSE>(p, it, hk, next, nwork, per_c, nHG, btf, cf, dtr, ready, sm.XS[q],
                     sm.XS[q ^ 1], sm.cs[q], sm.dt[q], sm.wtot[q], sm.vf[q], sm.w[q], sm.cs[q ^ 1], sm.dt[q ^ 1],
                     sm.wtot[q ^ 1], sm.vf[q ^ 1], sm.w[q ^ 1], s_gr, s_hb, &sm.ticket, A_logp, Dp, biasp, sm.wn);
        q ^= 1;
    }
    if (next >= nwork) break;
    work = next;
    }
}

template <int N>
hipError_t launch_n(const FusedParams& p, hipStream_t stream, hipEvent_t ev_begin, hipEvent_t ev_end)
{
    if (p.y32 && (p.vtab || p.z || p.norm_head)) return hipErrorInvalidValue;   // plain rows, no gate/norm
    if (p.vtab) {   // packed row: the chunk table first
        hipError_t e = launch_seq_table(p.seq_idx, p.arg_starts, p.T, p.nseq, kQ, p.nC, p.ring_rows, p.starts,
                                        p.vtab, nullptr, p.vcount, stream);
        if (e == hipSuccess && p.vorder) {
            hipLaunchKernelGGL((k_seq_order<kQ>), dim3(1), dim3(kTabThreads), 0, stream, p.vtab, p.starts, p.vcount,
                               static_cast<int>(p.T), p.vorder);
            e = hipGetLastError();
        }
        if (e != hipSuccess) return e;
    }
    int dev = 0, cus = 0;
    hipError_t err = hipGetDevice(&dev);
    if (err == hipSuccess) err = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (err != hipSuccess) return err;
    // four prep workgroups per (chunk, group) while that fills the chip at most
    // twice over; else two or one, each taking several parts with B loaded once
    const int64_t pairs = p.nC * p.b * p.G;
    const unsigned gz = pairs * kGramParts <= 2 * cus ? kGramParts : (pairs * 2 <= 2 * cus ? 2 : 1);
    const dim3 g_prep(static_cast<unsigned>(p.nC), static_cast<unsigned>(p.b * p.G), gz);
    if (p.vtab)
        hipLaunchKernelGGL((k_fused_prep<N, true>), g_prep, dim3(kPrepThreads), 0, stream, p);
    else
        hipLaunchKernelGGL((k_fused_prep<N, false>), g_prep, dim3(kPrepThreads), 0, stream, p);
    err = hipGetLastError();
    if (err == hipSuccess && ev_begin) err = hipEventRecord(ev_begin, stream);
    if (err != hipSuccess) return err;
    const int64_t nwork = p.nC * p.b * (p.H / p.HG);
    // one persistent workgroup per compute unit (the LDS footprint allows one);
    // p.max_workgroups caps it (a test setting: few workgroups, many items each)
    int64_t grid = nwork < cus ? nwork : cus;
    if (p.max_workgroups >= 1 && p.max_workgroups < grid) grid = p.max_workgroups;
    const dim3 g_main(static_cast<unsigned>(grid));
    const float* A_logp = p.A_log;
    const float* Dp = p.D;
    const float* biasp = p.dtx.bias;
    if (p.y32 && p.early_flag)
        hipLaunchKernelGGL((k_fused_main<N, false, true, true, false>), g_main, dim3(kMainThreads), 0, stream, p, A_logp, Dp,
                           biasp);
    else if (p.y32)
        hipLaunchKernelGGL((k_fused_main<N, false, false, true, false>), g_main, dim3(kMainThreads), 0, stream, p, A_logp,
                           Dp, biasp);
    else if (p.vtab && p.early_flag)
        hipLaunchKernelGGL((k_fused_main<N, true, true, false, false>), g_main, dim3(kMainThreads), 0, stream, p, A_logp, Dp,
                           biasp);
    else if (p.vtab && p.fuse_rf)
        hipLaunchKernelGGL((k_fused_main<N, true, false, false, true>), g_main, dim3(kMainThreads), 0, stream, p, A_logp,
                           Dp, biasp);
    else if (p.vtab)
        hipLaunchKernelGGL((k_fused_main<N, true, false, false, false>), g_main, dim3(kMainThreads), 0, stream, p, A_logp,
                           Dp, biasp);
    else if (p.early_flag)
        hipLaunchKernelGGL((k_fused_main<N, false, true, false, false>), g_main, dim3(kMainThreads), 0, stream, p, A_logp,
                           Dp, biasp);
    else if (p.fuse_rf)
        hipLaunchKernelGGL((k_fused_main<N, false, false, false, true>), g_main, dim3(kMainThreads), 0, stream, p,
                           A_logp, Dp, biasp);
    else
        hipLaunchKernelGGL((k_fused_main<N, false, false, false, false>), g_main, dim3(kMainThreads), 0, stream, p,
                           A_logp, Dp, biasp);
    err = hipGetLastError();
    if (err == hipSuccess && ev_end) err = hipEventRecord(ev_end, stream);
    return err;
}

}  // namespace

hipError_t launch_seq_table(const int32_t* seq_idx, const SeqStartsArg* arg_starts, int64_t T, int64_t nseq, int Q,
                            int64_t cap, int64_t ring_rows, int* starts, int4* vtab, int* seq_first, int* vcount,
                            hipStream_t stream)
{
    const int Ti = static_cast<int>(T), ns = static_cast<int>(nseq);
    if (seq_idx)
        hipLaunchKernelGGL(k_seq_starts, dim3(static_cast<unsigned>((Ti + 255) / 256)), dim3(256), 0, stream,
                           seq_idx, Ti, ns, starts);
    else
        hipLaunchKernelGGL(k_seq_starts_args, dim3(1), dim3(256), 0, stream, *arg_starts, starts);
    const int capi = static_cast<int>(cap), ring = static_cast<int>(ring_rows < 1 ? 1 : ring_rows);
    if (Q == kQ)
        hipLaunchKernelGGL((k_seq_chunks<kQ>), dim3(1), dim3(kTabThreads), 0, stream, starts, Ti, ns, capi, ring,
                           vtab, seq_first, vcount);
    else if (Q == 64)
        hipLaunchKernelGGL((k_seq_chunks<64>), dim3(1), dim3(kTabThreads), 0, stream, starts, Ti, ns, capi, ring,
                           vtab, seq_first, vcount);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

bool fused_supported(int64_t P, int64_t N, int64_t Q, bool bf16)
{
    return bf16 && P == kP && Q == kQ && (N == 64 || N == 128 || N == 256);
}

FusedLayout fused_layout(int64_t b, int64_t T, int64_t H, int64_t N, int64_t G, int64_t nC, int64_t nseq)
{
    auto al = [](size_t v) { return (v + 255) / 256 * 256; };
    FusedLayout w;
    // A packed row cut at its sequence starts has at most nC + nseq - 1 chunks
    // (and no more than T); only sequences longer than one chunk pass a state
    // between chunks, and there are fewer of them than chunks.
    w.nC = nseq > 0 ? std::min(nC + nseq - 1, T) : nC;
    w.ring_rows = nseq > 0 ? std::min(nseq, nC) : b;
    size_t off = kWorkspaceHeader;   // the status word sits in the header
    w.gram = off;
    off = al(off + sizeof(u16) * static_cast<size_t>(b * G * w.nC) * kTiles * 256);
    w.BT = off;
    off = al(off + sizeof(u16) * static_cast<size_t>(b * G * w.nC) * static_cast<size_t>(N * kQ));
    w.ring = off;
    off = al(off + sizeof(float) * static_cast<size_t>(w.ring_rows * H) * 2 * kP * static_cast<size_t>(N));
    w.flags = off;
    off = al(off + sizeof(int) * static_cast<size_t>(b * H * w.nC));
    w.ticket = off;
    off = al(off + 4 * sizeof(int));   // ticket, (unused), table entries
    w.starts = off;
    off = al(off + sizeof(int) * static_cast<size_t>(nseq > 0 ? nseq + 1 : 0));
    w.vtab = off;
    off = al(off + sizeof(int4) * static_cast<size_t>(nseq > 0 ? w.nC : 0));
    w.vorder = off;
    off = al(off + sizeof(int) * static_cast<size_t>(nseq > 0 ? w.nC : 0));
    w.total = off;
    return w;
}

hipError_t launch_fused(const FusedParams& p, hipStream_t stream, hipEvent_t ev_begin,
                        hipEvent_t ev_end)
{
    return p.N == 64    ? launch_n<64>(p, stream, ev_begin, ev_end)
           : p.N == 128 ? launch_n<128>(p, stream, ev_begin, ev_end)
                        : launch_n<256>(p, stream, ev_begin, ev_end);
}

}  // namespace ssd
