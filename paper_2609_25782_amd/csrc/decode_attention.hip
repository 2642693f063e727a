// Split-K paged grouped-query decode attention for gfx950 (data path 1 of the
// hot-cold hierarchy: every decode step reads the whole hot set).
//
// Work split.  A unit is one page (16 tokens) of one (row b, group of L KV
// heads); the units of all rows are laid end to end and cut into equal ranges,
// one per worker of a persistent grid, so long and short contexts balance
// exactly.  A worker is L consecutive waves, wave w taking KV head L hg + w of
// head group hg: with L = 4 the four waves of a worker read the four heads'
// tiles of each page side by side, which HBM serves faster than as many
// unrelated pages (DRAM row locality); L = 1 when the KV heads do not come in
// fours.  Where a worker's range meets the units of one (b, hg), each of its
// waves produces a partial result (running max m, weight sum l, unnormalised
// output o) for the query heads sharing its KV head; the combine kernel merges
// the partials of each (b, g) with the usual log-sum-exp rescaling.  Reduction
// order depends only on seq_lens, never on page placement, so results are
// bitwise independent of where pages sit in the pool.
//
// One wave processes one page of one KV head per step with matrix cores:
//   scores  S^T[t][h] = K[t][:] . Q[h][:]   v_mfma_f32_16x16x32_bf16 (f32: 16x16x4)
//           (16 tokens x 16 head slots; the group's heads fill the first slots)
//   output  O^T[d][h] += V^T[d][t] P^T[t][h] v_mfma_f32_16x16x16_bf16 (f32: 16x16x4)
// The score tile comes out of the first product in exactly the register layout
// the second product takes for P (lane l: head l % 16, tokens 4 (l / 16) + r),
// so the softmax needs no data movement besides two cross-lane max steps.
// Each query-head group reads every K/V byte once (the GQA reuse).
//
// Memory.  K tiles are stored as 16-byte groups of dims, token-minor, so the
// four 16-byte loads a lane issues for a K tile are each 1 KiB contiguous across
// the wave; V tiles are stored dims-major, token-minor, so each lane's slice of
// V^T for one 16-dim chunk is 8 contiguous bytes and a wave reads 512
// contiguous bytes per load.  Pages are addressed through buffer resources
// whose base is the page and whose size is its two tiles: an out-of-range page
// id becomes a zero-sized resource, reads return 0 and the row is flagged NaN.
// Each wave keeps a ring of page buffers in registers: while one page is
// computed, the loads of the next ring - 1 pages are in flight.

#include "device_common.h"
#include "kernels.h"

#include <math.h>

namespace hck {
namespace {

constexpr int kRsrcWord3 = 0x00020000;  // raw buffer, 32-bit data format (gfx9 family)

// Cache-policy bits of the K/V page loads: 2 = nontemporal (streaming).  Every
// K/V byte is read exactly once per call, so keeping it out of the caches'
// normal replacement leaves them to page ids, queries and partials.
#ifndef HCK_DECODE_LOAD_AUX
#define HCK_DECODE_LOAD_AUX 2
#endif
#ifndef HCK_RING_BF16_D128
#define HCK_RING_BF16_D128 3
#endif
// Waves per block of the split kernel.
#ifndef HCK_SPLIT_BLOCK_WAVES
#define HCK_SPLIT_BLOCK_WAVES 4
#endif
constexpr int kSplitBlockWaves = HCK_SPLIT_BLOCK_WAVES;
constexpr int kSplitBlockThreads = kSplitBlockWaves * kWave;

template <int D, bool BF16>
struct Shape {
    static constexpr int kElt = BF16 ? 2 : 4;
    static constexpr int kTile = kPageTokens * D * kElt;  // bytes of a K or V tile
    static constexpr int kKLoads = kTile / 1024;          // 16-byte K loads per lane
    static constexpr int kChunks = D / 16;                // 16-dim output chunks
};

template <bool BF16>
struct VSlice;
template <>
struct VSlice<true> {
    typedef u32x2 type;  // 4 bf16 tokens of one dim
};
template <>
struct VSlice<false> {
    typedef u32x4 type;  // 4 f32 tokens of one dim
};

template <int D, bool BF16>
struct PageRegs {
    u32x4 k[Shape<D, BF16>::kKLoads];
    typename VSlice<BF16>::type v[Shape<D, BF16>::kChunks];
};

__device__ __forceinline__ float wave_max_4(float x) {
    // max over lanes l, l^16, l^32, l^48 (the four token quarters of one head)
    x = fmaxf(x, __shfl_xor(x, 16));
    x = fmaxf(x, __shfl_xor(x, 32));
    return x;
}

__device__ __forceinline__ float wave_sum_4(float x) {
    x += __shfl_xor(x, 16);
    x += __shfl_xor(x, 32);
    return x;
}

// Where a piece's pages live, already offset to its layer and KV head: hot
// pages, and for tiered entries the cold pool and this layer's staging slots.
struct PageSrc {
    const char* hot = nullptr;
    const char* cold = nullptr;
    const char* stage = nullptr;
    int64_t hot_stride = 0, cold_stride = 0, slice_bytes = 0;
    unsigned num_hot = 0, num_cold = 0, num_stage = 0;
};

// Page ids are wave-uniform, so the tier choice is scalar.  An id outside its
// pool (or a negative entry) reads nothing: the buffer resource gets no records
// and the row is marked bad (NaN).
template <int D, bool BF16, bool TIERED>
__device__ __forceinline__ void load_page(PageRegs<D, BF16>& r, const PageSrc& ps, int pid, bool& bad,
                                          unsigned koff, unsigned voff) {
    using S = Shape<D, BF16>;
    const char* lh_base = ps.hot;
    int64_t stride = ps.hot_stride;
    unsigned n = ps.num_hot;
    unsigned id = static_cast<unsigned>(pid);
    if constexpr (TIERED) {
        const unsigned tag = id >> 29;  // 0 hot, 1 staged, 2 cold, otherwise invalid
        id &= static_cast<unsigned>(kPageIdMask);
        if (tag == 1) {
            lh_base = ps.stage;
            stride = ps.slice_bytes;
            n = ps.num_stage;
        } else if (tag == 2) {
            lh_base = ps.cold;
            stride = ps.cold_stride;
            n = ps.num_cold;
        } else if (tag != 0) {
            n = 0;
        }
    }
    const bool ok = id < n;
    bad |= !ok;
    const char* base = lh_base + static_cast<int64_t>(ok ? id : 0) * stride;
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(base), static_cast<short>(0),
                                          ok ? 2 * S::kTile : 0, kRsrcWord3);
#pragma unroll
    for (int i = 0; i < S::kKLoads; ++i)
        r.k[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, koff + 1024u * i, 0, HCK_DECODE_LOAD_AUX);
#pragma unroll
    for (int c = 0; c < S::kChunks; ++c) {
        if constexpr (BF16)
            r.v[c] = __builtin_amdgcn_raw_buffer_load_b64(rs, voff + S::kTile + 512u * c, 0, HCK_DECODE_LOAD_AUX);
        else
            r.v[c] = __builtin_amdgcn_raw_buffer_load_b128(rs, voff + S::kTile + 1024u * c, 0, HCK_DECODE_LOAD_AUX);
    }
}

// S^T tile of one page: lane l gets scores of head l % 16 for tokens 4 (l / 16) + r.
// Two accumulators halve the dependent MFMA chain; their sum is added once.
template <int D, bool BF16>
__device__ __forceinline__ f32x4 page_scores(const PageRegs<D, BF16>& r,
                                             const u32x4 (&q)[Shape<D, BF16>::kKLoads]) {
    using S = Shape<D, BF16>;
    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < S::kKLoads; ++i) {
        f32x4& acc = (i & 1) ? s1 : s0;
        if constexpr (BF16) {
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, r.k[i]),
                                                          __builtin_bit_cast(bf16x8, q[i]), acc, 0,
                                                          0, 0);
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j)
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(r.k[i][j]),
                                                           __uint_as_float(q[i][j]), acc, 0, 0, 0);
        }
    }
    return s0 + s1;
}

// Zero the V slice entries of tokens >= valid (this lane holds tokens 4 qg + j).
template <int D, bool BF16>
__device__ __forceinline__ void mask_v(PageRegs<D, BF16>& r, int valid, int qg) {
    using S = Shape<D, BF16>;
    const int t0 = 4 * qg;
    if constexpr (BF16) {
        const unsigned m0 = (t0 + 0 < valid ? 0x0000FFFFu : 0u) | (t0 + 1 < valid ? 0xFFFF0000u : 0u);
        const unsigned m1 = (t0 + 2 < valid ? 0x0000FFFFu : 0u) | (t0 + 3 < valid ? 0xFFFF0000u : 0u);
#pragma unroll
        for (int c = 0; c < S::kChunks; ++c) {
            r.v[c][0] &= m0;
            r.v[c][1] &= m1;
        }
    } else {
#pragma unroll
        for (int c = 0; c < S::kChunks; ++c)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (t0 + j >= valid) r.v[c][j] = 0u;
    }
}

template <int D, bool BF16>
struct SegmentState {
    u32x4 q[Shape<D, BF16>::kKLoads];
    f32x4 o[Shape<D, BF16>::kChunks];
    float m;
    float l;
};

// Online-softmax update and weighted V for one page with `valid` tokens (1..16).
template <int D, bool BF16>
__device__ __forceinline__ void compute_page(SegmentState<D, BF16>& st, PageRegs<D, BF16>& pg,
                                             int valid, float scale_log2, int qg) {
    using S = Shape<D, BF16>;
    f32x4 s = page_scores<D, BF16>(pg, st.q);
    if (valid < kPageTokens) {
#pragma unroll
        for (int r = 0; r < 4; ++r) s[r] = (4 * qg + r < valid) ? s[r] : -INFINITY;
        mask_v<D, BF16>(pg, valid, qg);
    }
    float mx = -INFINITY;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        s[r] *= scale_log2;
        mx = fmaxf(mx, s[r]);
    }
    // The running max m is the same on the four lanes of a head.  Only when some
    // lane sees a score above it is the page max reduced across lanes and the
    // accumulators rescaled; otherwise the reduced max would equal m and every
    // factor would be exactly 1, so skipping is bitwise identical.
    if (__builtin_amdgcn_ballot_w64(mx > st.m)) {
        const float m_new = fmaxf(st.m, wave_max_4(mx));
        const float alpha = __builtin_amdgcn_exp2f(st.m - m_new);
        st.l *= alpha;
#pragma unroll
        for (int c = 0; c < S::kChunks; ++c) st.o[c] *= alpha;
        st.m = m_new;
    }
    float p[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) p[r] = __builtin_amdgcn_exp2f(s[r] - st.m);
    if constexpr (BF16) {
        __bf16 pb[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            pb[r] = static_cast<__bf16>(p[r]);
            st.l += static_cast<float>(pb[r]);
        }
        const s16x4 pv = {__builtin_bit_cast(short, pb[0]), __builtin_bit_cast(short, pb[1]),
                          __builtin_bit_cast(short, pb[2]), __builtin_bit_cast(short, pb[3])};
#pragma unroll
        for (int c = 0; c < S::kChunks; ++c)
            st.o[c] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4, pg.v[c]),
                                                                pv, st.o[c], 0, 0, 0);
    } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) st.l += p[r];
#pragma unroll
        for (int c = 0; c < S::kChunks; ++c)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                st.o[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                    __uint_as_float(pg.v[c][j]), p[j], st.o[c], 0, 0, 0);
    }
}

// Fused merge: the split's partials cross between XCDs as device-scope
// stores and loads (cache-policy bit SC1 on gfx950).  The L2 of each XCD
// writes such stores through and does not serve such loads from its own
// lines, so neither the arrival nor the merge needs a whole-L2 write-back
// or invalidate.
constexpr int kScopeDevice = 16;  // SC1: device-scope coherence

// The workspace's partials through one buffer resource (offsets from part_o).
struct PartialsRsrc {
    __amdgpu_buffer_rsrc_t rs;
    const char* base;
    __device__ explicit PartialsRsrc(const DecodeArgs& a) : base(reinterpret_cast<const char*>(a.part_o)) {
        rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(a.part_o), static_cast<short>(0), 0x7FFFFFFF,
                                               kRsrcWord3);
    }
    __device__ unsigned off(const float* p) const {
        return static_cast<unsigned>(reinterpret_cast<const char*>(p) - base);
    }
    __device__ void store4(float* p, const f32x4& v) const {
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), rs, off(p), 0, kScopeDevice);
    }
    __device__ void store1(float* p, float v) const {
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), rs, off(p), 0, kScopeDevice);
    }
    __device__ f32x4 load4(const float* p) const {
        return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, off(p), 0, kScopeDevice));
    }
    __device__ float load1(const float* p) const {
        return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rs, off(p), 0, kScopeDevice));
    }
};

__device__ __forceinline__ void lse_merge(float& M, float& den, f32x4& acc, float m2, float l2,
                                          const f32x4& o2) {
    const float Mn = fmaxf(M, m2);
    const float c1 = (M == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(M - Mn);
    const float c2 = (m2 == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m2 - Mn);
    acc = acc * c1 + o2 * c2;
    den = den * c1 + l2 * c2;
    M = Mn;
}

// Range of waves whose partials belong to segment (b, g): units [u_a, u_a + nb).
struct SegWaves {
    int k_first, k_last, pieces;
};

__device__ __forceinline__ SegWaves seg_waves(int64_t u_a, int nb, int64_t T, int N) {
    SegWaves w;
    w.k_first = static_cast<int>(((u_a + 1) * N - 1) / T);
    w.k_last = static_cast<int>(((u_a + nb) * N - 1) / T);
    // with more waves than units every non-empty wave holds exactly one unit
    w.pieces = (N <= T) ? (w.k_last - w.k_first + 1) : nb;
    return w;
}

// One wave merges every query head of segment (b, g): lane l owns the items
// (head, 4-dim quad) l, l + 64, ...; loads of all its items for one partial
// are issued together.
template <int D, bool BF16>
__device__ __forceinline__ void store_quad(const DecodeArgs& a, int64_t orow, const f32x4& res) {
    if constexpr (BF16) {
        __bf16 v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) v[j] = static_cast<__bf16>(res[j]);
        *reinterpret_cast<u32x2*>(static_cast<__bf16*>(a.out) + orow) = __builtin_bit_cast(u32x2, v);
    } else {
        *reinterpret_cast<f32x4*>(static_cast<float*>(a.out) + orow) = res;
    }
}

// Every query head of (b, g) set to one value (rows with no pages, bad rows).
template <int D, bool BF16>
__device__ void fill_segment(const DecodeArgs& a, int b, int g, float value, int lane) {
    constexpr int kQuads = D / 4;
    for (int idx = lane; idx < a.group * kQuads; idx += kWave) {
        const int h = idx / kQuads, quad = idx % kQuads;
        store_quad<D, BF16>(a, (static_cast<int64_t>(b) * a.num_q_heads + g * a.group + h) * D + 4 * quad,
                            f32x4{value, value, value, value});
    }
}

template <int D, bool BF16>
__device__ void combine_segment(const DecodeArgs& a, int b, int g, int64_t u_a, int nb, int64_t T,
                                int lane) {
    const PartialsRsrc pr(a);
    constexpr int kQuads = D / 4;
    constexpr int kMaxItems = (16 * kQuads + kWave - 1) / kWave;
    constexpr int kBatch = 4;  // partials whose loads are in flight together
    const int items = a.group * kQuads;
    const int gw = a.group_waves;
    const int64_t sseg = static_cast<int64_t>(b) * (a.num_kv_heads / gw) + g / gw;
    const int w = g % gw;
    const int N = a.waves / gw;
    // fewer workers than units: workers k_first.. each hold one piece; more:
    // each unit is a piece, held by the worker that owns it
    const bool per_unit = N > T;
    const int k_first = static_cast<int>(((u_a + 1) * N - 1) / T);
    const int count = per_unit ? nb : static_cast<int>(((u_a + nb) * N - 1) / T) - k_first + 1;
    float M[kMaxItems], den[kMaxItems];
    f32x4 acc[kMaxItems];
#pragma unroll
    for (int it = 0; it < kMaxItems; ++it) {
        M[it] = -INFINITY;
        den[it] = 0.f;
        acc[it] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    for (int i0 = 0; i0 < count; i0 += kBatch) {
        float mk[kBatch][kMaxItems], lk[kBatch][kMaxItems];
        f32x4 ok[kBatch][kMaxItems];
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
            const int i = i0 + j < count ? i0 + j : count - 1;  // past the end: reload the last, unused
            const int k = per_unit ? static_cast<int>(((u_a + i + 1) * N - 1) / T) : k_first + i;
            const int64_t slot = (static_cast<int64_t>(k) + sseg) * gw + w;
            const float* pml = a.part_ml + slot * 2 * a.group;
#pragma unroll
            for (int it = 0; it < kMaxItems; ++it) {
                const int idx = it * kWave + lane;
                if (idx < items) {
                    const int h = idx / kQuads, quad = idx % kQuads;
                    mk[j][it] = pr.load1(pml + h);
                    lk[j][it] = pr.load1(pml + a.group + h);
                    ok[j][it] = pr.load4(a.part_o + (slot * a.group + h) * D + 4 * quad);
                }
            }
        }
#pragma unroll
        for (int j = 0; j < kBatch; ++j)
            if (i0 + j < count)
#pragma unroll
                for (int it = 0; it < kMaxItems; ++it)
                    if (it * kWave + lane < items)
                        lse_merge(M[it], den[it], acc[it], mk[j][it], lk[j][it], ok[j][it]);
    }
    const int32_t len = a.seq_lens[b];
    const bool invalid = static_cast<int64_t>(len) > kPageTokens * a.pt_stride;
    const float nan = __builtin_nanf("");
#pragma unroll
    for (int it = 0; it < kMaxItems; ++it) {
        const int idx = it * kWave + lane;
        if (idx < items) {
            const int h = idx / kQuads, quad = idx % kQuads;
            const f32x4 res = invalid ? f32x4{nan, nan, nan, nan} : acc[it] / den[it];
            store_quad<D, BF16>(a, (static_cast<int64_t>(b) * a.num_q_heads + g * a.group + h) * D + 4 * quad,
                                res);
        }
    }
}

// Fused append (paged_decode_attention_append): the piece holding a row's last
// page first writes the row's new token, k_new / v_new row b for this wave's
// KV head, into that page at slot (L - 1) % 16, then orders those stores before
// its own loads of the page (the same wave is the only reader of that page's
// tiles for this KV head in the launch).  Rows with L <= 0 or an invalid L, and
// tail entries that name no page (or a staging slot), write nothing.
template <int D, bool BF16, bool TIERED>
__device__ __forceinline__ void append_new_token(const DecodeArgs& a, const PageSrc& ps, const int32_t* row,
                                                 const Piece& pc, int nb, int seq_len, int lane) {
    using S = Shape<D, BF16>;
    if (!a.k_new || pc.p1 != nb || seq_len <= 0 || a.seq_lens[pc.b] != seq_len) return;
    unsigned id = static_cast<unsigned>(__builtin_amdgcn_readfirstlane(row[nb - 1]));
    const char* base = ps.hot;
    int64_t stride = ps.hot_stride;
    unsigned n = ps.num_hot;
    if constexpr (TIERED) {
        const unsigned tag = id >> 29;  // 0 hot, 2 cold; a staged slot is a copy, not the page
        id &= static_cast<unsigned>(kPageIdMask);
        if (tag == 2) {
            base = ps.cold;
            stride = ps.cold_stride;
            n = ps.num_cold;
        } else if (tag != 0) {
            n = 0;
        }
    }
    if (id >= n) return;
    char* lh = const_cast<char*>(base) + static_cast<int64_t>(id) * stride;
    const int slot = (seq_len - 1) % kPageTokens;
    const int64_t src = (static_cast<int64_t>(pc.b) * a.num_kv_heads + pc.g) * D * S::kElt;
    const char* ks = static_cast<const char*>(a.k_new) + src;
    const char* vs = static_cast<const char*>(a.v_new) + src;
    constexpr int x = 16 / S::kElt;  // elements per 16-byte group of the K tile
    if (lane < D / x)
        *reinterpret_cast<u32x4*>(lh + (static_cast<int64_t>(lane) * kPageTokens + slot) * 16) =
            *reinterpret_cast<const u32x4*>(ks + 16 * lane);
    for (int d = lane; d < D; d += kWave) {
        char* vd = lh + S::kTile + (static_cast<int64_t>(d) * kPageTokens + slot) * S::kElt;
        if constexpr (BF16)
            *reinterpret_cast<unsigned short*>(vd) = reinterpret_cast<const unsigned short*>(vs)[d];
        else
            *reinterpret_cast<unsigned*>(vd) = reinterpret_cast<const unsigned*>(vs)[d];
    }
    // Other lanes of this wave read these bytes back with the page's loads.  A
    // workgroup-scope release/acquire orders that in the memory model; waiting
    // for the stores to be acknowledged makes the order independent of how the
    // L1 treats the nontemporal loads (once per row's tail page: negligible).
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

__device__ __forceinline__ int load_ids(const int32_t* __restrict__ row, int first, int end,
                                        int lane) {
    const int i = first + lane;
    return i < end ? row[i] : -1;
}

// Process pages [p0, p1) of row b, KV head g, and write the partial to its slot.
// R page buffers form a ring: while one page is computed, the next R - 1 are
// in flight.
template <int D, bool BF16, int R, bool TIERED>
__device__ void run_piece(const DecodeArgs& a, const Piece& pc, int nb, int seq_len, bool row_invalid,
                          int lane, int64_t seg_first_unit, int64_t total_units) {
    using S = Shape<D, BF16>;
    const int h = lane & 15, qg = lane >> 4;
    const bool hvalid = h < a.group;
    SegmentState<D, BF16> st;
    {
        const char* qrow = static_cast<const char*>(a.q) +
                           (static_cast<int64_t>(pc.b) * a.num_q_heads + pc.g * a.group +
                            (hvalid ? h : 0)) * D * S::kElt;
#pragma unroll
        for (int i = 0; i < S::kKLoads; ++i)
            st.q[i] = hvalid ? *reinterpret_cast<const u32x4*>(qrow + 16 * (4 * i + qg))
                             : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int c = 0; c < S::kChunks; ++c) st.o[c] = f32x4{0.f, 0.f, 0.f, 0.f};
    st.m = -INFINITY;
    st.l = 0.f;
    bool bad = false;

    const int32_t* row = a.page_table + static_cast<int64_t>(pc.b) * a.pt_stride;
    const int64_t head_off = static_cast<int64_t>(pc.g) * 2 * S::kTile;
    PageSrc ps;
    ps.hot = a.hot + head_off;
    ps.hot_stride = a.hot_stride;
    ps.num_hot = static_cast<unsigned>(a.num_pages);
    if constexpr (TIERED) {
        ps.cold = a.cold + head_off;
        ps.cold_stride = a.cold_stride;
        ps.stage = a.stage + head_off;
        ps.slice_bytes = a.slice_bytes;
        ps.num_cold = static_cast<unsigned>(a.num_cold_pages);
        ps.num_stage = static_cast<unsigned>(a.num_stage_slots);
    }
    append_new_token<D, BF16, TIERED>(a, ps, row, pc, nb, seq_len, lane);
    const unsigned koff = 16u * lane;
    const unsigned voff = BF16 ? (32u * (lane & 15) + 8u * qg) : (64u * (lane & 15) + 16u * qg);
    // valid tokens of the row's last page (16 when full)
    const int tail_valid = seq_len - kPageTokens * (nb - 1);

    int ids_cur = load_ids(row, pc.p0, pc.p1, lane);
    int ids_nxt = load_ids(row, pc.p0 + kWave, pc.p1, lane);
    int cur_chunk = 0;
    auto pid_at = [&](int i) -> int {
        const int rel = i - pc.p0;
        const int cc = rel >> 6;
        if (cc != cur_chunk) {
            ids_cur = ids_nxt;
            cur_chunk = cc;
            ids_nxt = load_ids(row, pc.p0 + kWave * (cc + 1), pc.p1, lane);
        }
        return __builtin_amdgcn_readlane(ids_cur, rel & 63);
    };

    PageRegs<D, BF16> buf[R];
#pragma unroll
    for (int r = 0; r < R - 1; ++r)
        if (pc.p0 + r < pc.p1)
            load_page<D, BF16, TIERED>(buf[r], ps, pid_at(pc.p0 + r), bad, koff, voff);
    for (int i = pc.p0; i < pc.p1; i += R) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int ip = i + r;
            if (ip < pc.p1) {
                const int ahead = ip + R - 1;
                if (ahead < pc.p1)
                    load_page<D, BF16, TIERED>(buf[(r + R - 1) % R], ps, pid_at(ahead), bad, koff, voff);
                compute_page<D, BF16>(st, buf[r], ip == nb - 1 ? tail_valid : kPageTokens,
                                      a.scale_log2, qg);
            }
        }
    }

    float l = wave_sum_4(st.l);
    if (bad) l = __builtin_nanf("");
    if (pc.p0 == 0 && pc.p1 == nb) {
        // The piece is the whole segment: its normalised result is the output.
        // (o + 0) / l is what merging this one partial gives, bit for bit.
        if (hvalid) {
            const float nan = __builtin_nanf("");
            const int64_t orow = (static_cast<int64_t>(pc.b) * a.num_q_heads + pc.g * a.group + h) * D + 4 * qg;
#pragma unroll
            for (int c = 0; c < S::kChunks; ++c)
                store_quad<D, BF16>(a, orow + 16 * c,
                                    row_invalid ? f32x4{nan, nan, nan, nan} : (st.o[c] + 0.f) / l);
        }
        return;
    }
    if (hvalid) {
        float* po = a.part_o + (static_cast<int64_t>(pc.slot) * a.group + h) * D + 4 * qg;
        float* pml = a.part_ml + static_cast<int64_t>(pc.slot) * 2 * a.group;
        if (a.fused) {
            const PartialsRsrc pr(a);
#pragma unroll
            for (int c = 0; c < S::kChunks; ++c) pr.store4(po + 16 * c, st.o[c]);
            if (qg == 0) {
                pr.store1(pml + h, st.m);
                pr.store1(pml + a.group + h, l);
            }
        } else {
#pragma unroll
            for (int c = 0; c < S::kChunks; ++c) *reinterpret_cast<f32x4*>(po + 16 * c) = st.o[c];
            if (qg == 0) {
                pml[h] = st.m;
                pml[a.group + h] = l;
            }
        }
    }
    if (a.fused) {
        // The wave that delivers the last partial of (b, g) merges them all.
        const SegWaves sw = seg_waves(seg_first_unit, nb, total_units, a.waves / a.group_waves);
        int32_t* cnt = a.counters + pc.b * a.num_kv_heads + pc.g;
        int prev = 0;
        // The partials went out as device-scope stores: once this wave's are
        // acknowledged they are visible to every XCD, and the merging wave
        // reads them back with device-scope loads.
        __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
        if (lane == 0) prev = __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        prev = __builtin_amdgcn_readfirstlane(__shfl(prev, 0));
        if (prev + 1 == sw.pieces) {
            combine_segment<D, BF16>(a, pc.b, pc.g, seg_first_unit, nb, total_units, lane);
            if (lane == 0) __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);  // next call
        }
    }
}

// ---------------------------------------------------------------------------
// Vector-ALU variant (bf16, at most 8 query heads per KV head).  Same work
// split, page loads, partial format and combine as the matrix-core path; both
// products run as v_dot2_f32_bf16 instead.  It exists to measure the choice of
// matrix cores on the same memory schedule.
//
// Scores: lane (t = l % 16, qq = l / 16) holds a quarter of token t's dims (the
// K loads are shared with the matrix-core path), so it forms partial dot
// products for all 8 head slots from the group's queries in LDS, and a
// reduce-scatter over the quarters leaves lane (t, qq) with the full scores of
// heads 2 qq and 2 qq + 1.  The bf16 weights cross to the output layout through
// 256 bytes of LDS.  Output: lane (dl, qg) holds dims 16 c + dl of tokens
// 4 qg .. 4 qg + 3 for every chunk c (the V loads of the matrix-core path) and
// accumulates all 8 head slots over its tokens; the four token quarters are
// summed once per piece.
constexpr int kValuMaxGroup = 8;

template <int D>
struct ValuLds {
    u32x4 q[(D / 8) * kValuMaxGroup];  // [load i][head][quarter qq]: dims 8 (4 i + qq) .. + 7
    unsigned p[kPageTokens * 4];       // [token][qq]: bf16 weights of heads 2 qq, 2 qq + 1
};

template <int D>
struct ValuState {
    float o[kValuMaxGroup][D / 16];  // lane (dl, qg): head h, dim 16 c + dl, over tokens 4 qg .. + 3
    float m[2], l[2];                // lane (t, qq): heads 2 qq + e; l over token t only
};

// Order this wave's LDS accesses: earlier writes complete before later reads,
// and the compiler moves no LDS access across it.
__device__ __forceinline__ void wave_lds_sync() { __asm__ volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

__device__ __forceinline__ float dot2_bf16(unsigned a, unsigned b, float c) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b), c,
                                           false);
}

__device__ __forceinline__ float readlane_f(float x, int lane) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), lane));
}

template <int D>
__device__ __forceinline__ void compute_page_valu(ValuState<D>& st, PageRegs<D, true>& pg, int valid,
                                                  float scale_log2, int lane, ValuLds<D>& sm) {
    using S = Shape<D, true>;
    const int t = lane & 15, qq = lane >> 4, qg = lane >> 4;
    // partial scores of token t over this lane's dims, all 8 head slots
    float s[kValuMaxGroup];
#pragma unroll
    for (int h = 0; h < kValuMaxGroup; ++h) s[h] = 0.f;
#pragma unroll
    for (int i = 0; i < S::kKLoads; ++i) {
#pragma unroll
        for (int h = 0; h < kValuMaxGroup; ++h) {
            const u32x4 qv = sm.q[(i * kValuMaxGroup + h) * 4 + qq];
#pragma unroll
            for (int j = 0; j < 4; ++j) s[h] = dot2_bf16(pg.k[i][j], qv[j], s[h]);
        }
    }
    // reduce-scatter over the quarters: lanes l and l ^ 32 split heads 0-3 / 4-7,
    // then lanes l and l ^ 16 split each half in pairs
    const bool upper = lane >= 32, odd = (lane & 16) != 0;
    float k4[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const float send = upper ? s[j] : s[4 + j];
        k4[j] = (upper ? s[4 + j] : s[j]) + __shfl_xor(send, 32);
    }
    float sh[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
        const float send = odd ? k4[e] : k4[2 + e];
        sh[e] = (odd ? k4[2 + e] : k4[e]) + __shfl_xor(send, 16);
    }
    // online softmax for heads 2 qq + e at token t (same lazy rescale as above)
#pragma unroll
    for (int e = 0; e < 2; ++e) sh[e] = t < valid ? sh[e] * scale_log2 : -INFINITY;
    if (__builtin_amdgcn_ballot_w64(sh[0] > st.m[0] || sh[1] > st.m[1])) {
        float mx[2] = {sh[0], sh[1]};
#pragma unroll
        for (int o = 1; o < 16; o <<= 1)
#pragma unroll
            for (int e = 0; e < 2; ++e) mx[e] = fmaxf(mx[e], __shfl_xor(mx[e], o));
        float alpha[2];
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            const float mn = fmaxf(st.m[e], mx[e]);
            alpha[e] = __builtin_amdgcn_exp2f(st.m[e] - mn);
            st.l[e] *= alpha[e];
            st.m[e] = mn;
        }
#pragma unroll
        for (int h = 0; h < kValuMaxGroup; ++h) {
            const float ah = readlane_f(alpha[h & 1], 16 * (h >> 1));
#pragma unroll
            for (int c = 0; c < S::kChunks; ++c) st.o[h][c] *= ah;
        }
    }
    __bf16 pb[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
        pb[e] = static_cast<__bf16>(__builtin_amdgcn_exp2f(sh[e] - st.m[e]));
        st.l[e] += static_cast<float>(pb[e]);
    }
    sm.p[t * 4 + qq] = static_cast<unsigned>(__builtin_bit_cast(unsigned short, pb[0])) |
                       (static_cast<unsigned>(__builtin_bit_cast(unsigned short, pb[1])) << 16);
    wave_lds_sync();
    // w[j][hp] = weights of heads 2 hp, 2 hp + 1 at token 4 qg + j
    u32x4 w[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) w[j] = *reinterpret_cast<const u32x4*>(sm.p + 4 * (4 * qg + j));
    unsigned p01[kValuMaxGroup], p23[kValuMaxGroup];
#pragma unroll
    for (int hp = 0; hp < 4; ++hp) {
        p01[2 * hp] = (w[0][hp] & 0xFFFFu) | (w[1][hp] << 16);
        p01[2 * hp + 1] = (w[0][hp] >> 16) | (w[1][hp] & 0xFFFF0000u);
        p23[2 * hp] = (w[2][hp] & 0xFFFFu) | (w[3][hp] << 16);
        p23[2 * hp + 1] = (w[2][hp] >> 16) | (w[3][hp] & 0xFFFF0000u);
    }
    if (valid < kPageTokens) mask_v<D, true>(pg, valid, qg);
#pragma unroll
    for (int c = 0; c < S::kChunks; ++c)
#pragma unroll
        for (int h = 0; h < kValuMaxGroup; ++h) {
            st.o[h][c] = dot2_bf16(pg.v[c][0], p01[h], st.o[h][c]);
            st.o[h][c] = dot2_bf16(pg.v[c][1], p23[h], st.o[h][c]);
        }
    __asm__ volatile("" ::: "memory");  // the next page's weight writes stay after these reads
}

template <int D, int R, bool TIERED>
__device__ void run_piece_valu(const DecodeArgs& a, const Piece& pc, int nb, int seq_len, bool row_invalid,
                               int lane, ValuLds<D>& sm) {
    using S = Shape<D, true>;
    constexpr int kGroups = D / 8;
    // the group's queries (zero beyond `group` heads) into LDS
    wave_lds_sync();  // the previous piece's reads are done
    {
        const __bf16* qrow = static_cast<const __bf16*>(a.q) +
                             (static_cast<int64_t>(pc.b) * a.num_q_heads + pc.g * a.group) * D;
        for (int e = lane; e < kGroups * kValuMaxGroup; e += kWave) {
            const int h = e / kGroups, grp = e % kGroups;
            const u32x4 v = h < a.group ? *reinterpret_cast<const u32x4*>(qrow + h * D + 8 * grp)
                                        : u32x4{0u, 0u, 0u, 0u};
            sm.q[((grp >> 2) * kValuMaxGroup + h) * 4 + (grp & 3)] = v;
        }
    }
    wave_lds_sync();
    ValuState<D> st;
#pragma unroll
    for (int h = 0; h < kValuMaxGroup; ++h)
#pragma unroll
        for (int c = 0; c < S::kChunks; ++c) st.o[h][c] = 0.f;
    st.m[0] = st.m[1] = -INFINITY;
    st.l[0] = st.l[1] = 0.f;
    bool bad = false;

    const int32_t* row = a.page_table + static_cast<int64_t>(pc.b) * a.pt_stride;
    const int64_t head_off = static_cast<int64_t>(pc.g) * 2 * S::kTile;
    PageSrc ps;
    ps.hot = a.hot + head_off;
    ps.hot_stride = a.hot_stride;
    ps.num_hot = static_cast<unsigned>(a.num_pages);
    if constexpr (TIERED) {
        ps.cold = a.cold + head_off;
        ps.cold_stride = a.cold_stride;
        ps.stage = a.stage + head_off;
        ps.slice_bytes = a.slice_bytes;
        ps.num_cold = static_cast<unsigned>(a.num_cold_pages);
        ps.num_stage = static_cast<unsigned>(a.num_stage_slots);
    }
    append_new_token<D, true, TIERED>(a, ps, row, pc, nb, seq_len, lane);
    const int qg = lane >> 4;
    const unsigned koff = 16u * lane;
    const unsigned voff = 32u * (lane & 15) + 8u * qg;
    const int tail_valid = seq_len - kPageTokens * (nb - 1);

    int ids_cur = load_ids(row, pc.p0, pc.p1, lane);
    int ids_nxt = load_ids(row, pc.p0 + kWave, pc.p1, lane);
    int cur_chunk = 0;
    auto pid_at = [&](int i) -> int {
        const int rel = i - pc.p0;
        const int cc = rel >> 6;
        if (cc != cur_chunk) {
            ids_cur = ids_nxt;
            cur_chunk = cc;
            ids_nxt = load_ids(row, pc.p0 + kWave * (cc + 1), pc.p1, lane);
        }
        return __builtin_amdgcn_readlane(ids_cur, rel & 63);
    };

    PageRegs<D, true> buf[R];
#pragma unroll
    for (int r = 0; r < R - 1; ++r)
        if (pc.p0 + r < pc.p1) load_page<D, true, TIERED>(buf[r], ps, pid_at(pc.p0 + r), bad, koff, voff);
    for (int i = pc.p0; i < pc.p1; i += R) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int ip = i + r;
            if (ip < pc.p1) {
                const int ahead = ip + R - 1;
                if (ahead < pc.p1)
                    load_page<D, true, TIERED>(buf[(r + R - 1) % R], ps, pid_at(ahead), bad, koff, voff);
                compute_page_valu<D>(st, buf[r], ip == nb - 1 ? tail_valid : kPageTokens, a.scale_log2,
                                     lane, sm);
            }
        }
    }

    // outputs: reduce-scatter over the token quarters (lane (dl, qg) keeps heads
    // 2 qg, 2 qg + 1), then every lane writes its two heads' dims 16 c + dl
    const bool upper = lane >= 32, odd = (lane & 16) != 0;
    float o4[4][S::kChunks];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int c = 0; c < S::kChunks; ++c) {
            const float send = upper ? st.o[j][c] : st.o[4 + j][c];
            o4[j][c] = (upper ? st.o[4 + j][c] : st.o[j][c]) + __shfl_xor(send, 32);
        }
    float o2[2][S::kChunks];
#pragma unroll
    for (int e = 0; e < 2; ++e)
#pragma unroll
        for (int c = 0; c < S::kChunks; ++c) {
            const float send = odd ? o4[e][c] : o4[2 + e][c];
            o2[e][c] = (odd ? o4[2 + e][c] : o4[e][c]) + __shfl_xor(send, 16);
        }
    // weight sums: lane (t, qq) holds token t's share of heads 2 qq + e
    float l[2] = {st.l[0], st.l[1]};
#pragma unroll
    for (int o = 1; o < 16; o <<= 1)
#pragma unroll
        for (int e = 0; e < 2; ++e) l[e] += __shfl_xor(l[e], o);
    const int dl = lane & 15;
    if (pc.p0 == 0 && pc.p1 == nb) {
        // the whole segment: write its output (what merging one partial gives)
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            const int h = 2 * qg + e;
            if (h < a.group) {
                const float den = bad ? __builtin_nanf("") : l[e];
                __bf16* orow = static_cast<__bf16*>(a.out) +
                               (static_cast<int64_t>(pc.b) * a.num_q_heads + pc.g * a.group + h) * D + dl;
#pragma unroll
                for (int c = 0; c < S::kChunks; ++c)
                    orow[16 * c] = static_cast<__bf16>(row_invalid ? __builtin_nanf("") : (o2[e][c] + 0.f) / den);
            }
        }
        return;
    }
#pragma unroll
    for (int e = 0; e < 2; ++e) {
        const int h = 2 * qg + e;
        if (h < a.group) {
            float* po = a.part_o + (static_cast<int64_t>(pc.slot) * a.group + h) * D + dl;
#pragma unroll
            for (int c = 0; c < S::kChunks; ++c) po[16 * c] = o2[e][c];
            if (dl == 0) {
                float* pml = a.part_ml + static_cast<int64_t>(pc.slot) * 2 * a.group;
                pml[h] = st.m[e];
                pml[a.group + h] = bad ? __builtin_nanf("") : l[e];
            }
        }
    }
}

// Register budget of the split kernel: with HCK_SPLIT_WAVES_PER_EU = n the
// compiler keeps it within 512 / n registers so that n waves fit per SIMD.
#ifndef HCK_SPLIT_WAVES_PER_EU
#define HCK_SPLIT_WAVES_PER_EU 1
#endif

template <int D, bool BF16, int R, bool TIERED, bool VALU>
__global__ __launch_bounds__(kSplitBlockThreads)
__attribute__((amdgpu_waves_per_eu(HCK_SPLIT_WAVES_PER_EU))) void decode_split_kernel(DecodeArgs a) {
    extern __shared__ int32_t s_pref[];
    block_prefix_pages<kSplitBlockThreads>(a.seq_lens, a.batch, a.pt_stride, s_pref);
    __syncthreads();
    if (blockIdx.x == 0)  // the combine reads the row prefix instead of rescanning the lengths
        for (int b = threadIdx.x; b <= a.batch; b += kSplitBlockThreads) a.row_pref[b] = s_pref[b];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(blockIdx.x * kSplitBlockWaves + threadIdx.x / kWave);
    if (wave >= a.waves) return;
    // the worker this wave belongs to, and its KV head within the worker's head group
    const int gw = a.group_waves;
    const int heads = a.num_kv_heads / gw;
    const int worker = wave / gw, w_in = wave % gw;
    // rows with no pages get no pieces: write them here (0 for L = 0, NaN for L < 0)
    for (int seg = wave; seg < a.batch * a.num_kv_heads; seg += a.waves) {
        const int b = seg / a.num_kv_heads;
        const int32_t len = a.seq_lens[b];
        if (len <= 0)
            fill_segment<D, BF16>(a, b, seg % a.num_kv_heads, len == 0 ? 0.f : __builtin_nanf(""), lane);
    }
    const int64_t total = static_cast<int64_t>(lds_uniform(s_pref + a.batch)) * heads;
    int64_t u, u1;
    wave_units(total, worker, a.waves / gw, u, u1);
    // the segment (row, head group) whose first piece this worker holds and
    // whose other pieces belong to later workers: the combine merges it
    int32_t split_seg = -1;
    while (u < u1) {
        Piece pc = piece_at<true>(s_pref, a.batch, heads, worker, u, u1);
        if (pc.p1 <= pc.p0) break;  // cannot happen for a consistent prefix; never spin
        const int nb = lds_uniform(s_pref + pc.b + 1) - lds_uniform(s_pref + pc.b);
        const int32_t len = a.seq_lens[pc.b];
        const int seq_len = len < kPageTokens * nb ? len : kPageTokens * nb;
        const bool row_invalid = static_cast<int64_t>(len) > kPageTokens * a.pt_stride;
        if (pc.p0 == 0 && pc.p1 < nb) split_seg = pc.b * heads + pc.g;
        const int64_t seg_first = static_cast<int64_t>(lds_uniform(s_pref + pc.b)) * heads +
                                  static_cast<int64_t>(pc.g) * nb;
        const int span = pc.p1 - pc.p0;
        pc.g = pc.g * gw + w_in;
        pc.slot = pc.slot * gw + w_in;
        if constexpr (VALU) {
            __shared__ ValuLds<D> s_valu[kSplitBlockWaves];
            run_piece_valu<D, R, TIERED>(a, pc, nb, seq_len, row_invalid, lane, s_valu[threadIdx.x / kWave]);
        } else {
            run_piece<D, BF16, R, TIERED>(a, pc, nb, seq_len, row_invalid, lane, seg_first, total);
        }
        u += span;
    }
    if (!a.fused && w_in == 0 && lane == 0) a.split_segs[worker] = split_seg;
}

// Merge the partials of one (b, g) for one query head and write its output row.
// The D/4 lanes of a lane group each own four output dims, and lane groups take
// every stride-th partial; loads for four partials are issued before any of
// them is merged.  Narrow: one wave per (b, g, h), four heads per block.  Wide
// (many partials per segment, i.e. small batches): the block's four waves share
// one (b, g, h) and merge their results through LDS.  The partials of a segment
// are those of workers k_first..k_last when there are fewer workers than units,
// and one per unit (the worker that owns it) otherwise.  Only segments split
// over several workers have partials (the split writes the others' output
// itself): the grid walks either all segments, skipping the rest, or, when
// workers are fewer than segments, the workers' split-segment entries.
#ifndef HCK_WIDE_COMBINE_PIECES
#define HCK_WIDE_COMBINE_PIECES 12
#endif
constexpr int kWideCombinePieces = HCK_WIDE_COMBINE_PIECES;

template <int D, bool BF16, bool WIDE>
__global__ __launch_bounds__(kBlockThreads) void decode_combine_kernel(DecodeArgs a) {
    constexpr int kQuads = D / 4;
    constexpr int kGroups = kWave / kQuads;
    constexpr int kUnroll = 4;
    constexpr int kStride = WIDE ? kBlockWaves * kGroups : kGroups;
    __shared__ float s_merge[WIDE ? kBlockWaves : 1][kQuads][6];
    const int wave = threadIdx.x / kWave;
    const int Lw = a.group_waves;
    const int heads = a.num_kv_heads / Lw;
    int b, g, hy;
    if (a.combine_by_worker) {
        // blockIdx.x: a worker; blockIdx.y: (KV head within the head group, head block)
        const int32_t e = a.split_segs[blockIdx.x];
        if (e < 0) return;  // whole block
        const int ny = WIDE ? a.group : (a.group + kBlockWaves - 1) / kBlockWaves;
        b = e / heads;
        g = (e % heads) * Lw + static_cast<int>(blockIdx.y) / ny;
        hy = static_cast<int>(blockIdx.y) % ny;
    } else {
        b = static_cast<int>(blockIdx.x) / a.num_kv_heads;
        g = static_cast<int>(blockIdx.x) % a.num_kv_heads;
        hy = static_cast<int>(blockIdx.y);
    }
    const int h = WIDE ? hy : hy * kBlockWaves + wave;
    if (h >= a.group) return;  // never taken by a wide block: its grid has one block per head
    const int lane = threadIdx.x & (kWave - 1);
    const int quad = lane % kQuads, grp = lane / kQuads;
    const int gid = WIDE ? wave * kGroups + grp : grp;

    // pages of the rows before b, and of all rows (the split kernel's prefix)
    const int64_t before = a.row_pref[b], total = a.row_pref[a.batch];
    const int32_t len = a.seq_lens[b];
    const int nb = row_pages(len, a.pt_stride);
    // The split wrote rows with no pages and segments it did not split
    // (uniform over the block: a wide block holds one segment).
    if (nb == 0) return;
    const bool invalid = static_cast<int64_t>(len) > kPageTokens * a.pt_stride;
    // units of head group g / Lw over the workers' ranges; this head's partials
    // are slot (worker + b * heads + g / Lw) * Lw + g % Lw
    const int64_t sseg = static_cast<int64_t>(b) * heads + g / Lw;
    const int w_in = g % Lw;
    const int64_t T = total * heads;
    const int64_t u_a = before * heads + static_cast<int64_t>(g / Lw) * nb;
    const int N = a.waves / Lw;
    const int k_first = static_cast<int>(((u_a + 1) * N - 1) / T);
    const int k_last = static_cast<int>(((u_a + nb) * N - 1) / T);
    const bool per_unit = N > T;  // every non-empty wave holds exactly one unit
    const int count = per_unit ? nb : k_last - k_first + 1;
    if (count == 1) return;
    f32x4 res;
    float M = -INFINITY, den = 0.f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    if (!invalid) {
        for (int i0 = gid; i0 < count; i0 += kUnroll * kStride) {
            float mk[kUnroll], lk[kUnroll];
            f32x4 ok[kUnroll];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const int i = i0 + u * kStride;
                const int k = per_unit ? static_cast<int>(((u_a + i + 1) * N - 1) / T) : k_first + i;
                // waves whose own unit range is empty wrote nothing to their slot
                const bool use = i < count &&
                                 (per_unit || static_cast<int64_t>(k) * T / N != static_cast<int64_t>(k + 1) * T / N);
                const int64_t slot = (static_cast<int64_t>(use ? k : 0) + sseg) * Lw + w_in;
                const float* pml = a.part_ml + slot * 2 * a.group;
                const float m_raw = pml[h], l_raw = pml[a.group + h];
                const f32x4 o_raw =
                    *reinterpret_cast<const f32x4*>(a.part_o + (slot * a.group + h) * D + 4 * quad);
                mk[u] = use ? m_raw : -INFINITY;
                lk[u] = use ? l_raw : 0.f;
                ok[u] = use ? o_raw : f32x4{0.f, 0.f, 0.f, 0.f};
            }
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) lse_merge(M, den, acc, mk[u], lk[u], ok[u]);
        }
#pragma unroll
        for (int off = kQuads; off < kWave; off <<= 1) {
            const float M2 = __shfl_xor(M, off), den2 = __shfl_xor(den, off);
            f32x4 acc2;
#pragma unroll
            for (int j = 0; j < 4; ++j) acc2[j] = __shfl_xor(acc[j], off);
            lse_merge(M, den, acc, M2, den2, acc2);
        }
    }
    if constexpr (WIDE) {
        // the block's waves took disjoint partials: merge their results in LDS
        if (grp == 0) {
            float* e = s_merge[wave][quad];
            e[0] = M;
            e[1] = den;
#pragma unroll
            for (int j = 0; j < 4; ++j) e[2 + j] = acc[j];
        }
        __syncthreads();
        if (wave != 0) return;
#pragma unroll
        for (int w = 1; w < kBlockWaves; ++w) {
            const float* e = s_merge[w][quad];
            lse_merge(M, den, acc, e[0], e[1], f32x4{e[2], e[3], e[4], e[5]});
        }
    }
    if (invalid) {
        const float nan = __builtin_nanf("");
        res = f32x4{nan, nan, nan, nan};
    } else {
        res = acc / den;
    }
    if (grp == 0) {
        const int64_t orow =
            (static_cast<int64_t>(b) * a.num_q_heads + g * a.group + h) * D + 4 * quad;
        if constexpr (BF16) {
            __bf16 v[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] = static_cast<__bf16>(res[j]);
            *reinterpret_cast<u32x2*>(static_cast<__bf16*>(a.out) + orow) = __builtin_bit_cast(u32x2, v);
        } else {
            *reinterpret_cast<f32x4*>(static_cast<float*>(a.out) + orow) = res;
        }
    }
}

// Ring depth per shape: the deepest ring that still leaves two (or three)
// waves per SIMD, i.e. at most 256 (168) VGPRs.
template <int D, bool BF16>
constexpr int ring_depth() {
    return BF16 ? (D == 128 ? HCK_RING_BF16_D128 : 5) : (D == 128 ? 2 : 3);
}

template <int D, bool BF16, bool VALU>
const void* split_kernel_ptr(bool tiered) {
    constexpr int R = ring_depth<D, BF16>();
    return tiered ? reinterpret_cast<const void*>(&decode_split_kernel<D, BF16, R, true, VALU>)
                  : reinterpret_cast<const void*>(&decode_split_kernel<D, BF16, R, false, VALU>);
}

// The vector-ALU variant exists for bf16 only.
const void* pick_split(int head_dim, int dtype, bool tiered, bool valu) {
    if (dtype == kDtypeBf16) {
        if (head_dim == 128)
            return valu ? split_kernel_ptr<128, true, true>(tiered) : split_kernel_ptr<128, true, false>(tiered);
        if (head_dim == 64)
            return valu ? split_kernel_ptr<64, true, true>(tiered) : split_kernel_ptr<64, true, false>(tiered);
    } else if (!valu) {
        if (head_dim == 128) return split_kernel_ptr<128, false, false>(tiered);
        if (head_dim == 64) return split_kernel_ptr<64, false, false>(tiered);
    }
    return nullptr;
}

template <int D, bool BF16>
const void* combine_kernel_ptr(bool wide) {
    return wide ? reinterpret_cast<const void*>(&decode_combine_kernel<D, BF16, true>)
                : reinterpret_cast<const void*>(&decode_combine_kernel<D, BF16, false>);
}

const void* pick_combine(int head_dim, int dtype, bool wide) {
    if (dtype == kDtypeBf16) {
        if (head_dim == 128) return combine_kernel_ptr<128, true>(wide);
        if (head_dim == 64) return combine_kernel_ptr<64, true>(wide);
    } else {
        if (head_dim == 128) return combine_kernel_ptr<128, false>(wide);
        if (head_dim == 64) return combine_kernel_ptr<64, false>(wide);
    }
    return nullptr;
}

size_t prefix_lds_bytes(int batch) { return static_cast<size_t>(batch + 1) * sizeof(int32_t); }

}  // namespace

hipError_t launch_decode_split(const DecodeArgs& a, int head_dim, int dtype, hipStream_t s,
                               const LaunchEvents& ev) {
    if (a.valu && (a.group > kValuMaxGroup || a.fused)) return hipErrorInvalidValue;
    // a worker's waves must share a block and split the KV heads and waves evenly
    if (a.group_waves < 1 || kSplitBlockWaves % a.group_waves || a.num_kv_heads % a.group_waves ||
        a.waves % a.group_waves)
        return hipErrorInvalidValue;
    const void* k = pick_split(head_dim, dtype, a.tiered != 0, a.valu != 0);
    if (!k || a.waves <= 0) return hipErrorInvalidValue;
    const int blocks = (a.waves + kSplitBlockWaves - 1) / kSplitBlockWaves;
    void* args[] = {const_cast<DecodeArgs*>(&a)};
    return launch_kernel(k, dim3(blocks), dim3(kSplitBlockThreads), args, prefix_lds_bytes(a.batch), s, ev);
}

hipError_t launch_decode_combine(const DecodeArgs& a, int head_dim, int dtype, hipStream_t s,
                                 const LaunchEvents& ev) {
    const int segs = a.batch * a.num_kv_heads;
    if (segs == 0) return hipSuccess;
    if (a.group_waves < 1 || a.num_kv_heads % a.group_waves || a.waves % a.group_waves)
        return hipErrorInvalidValue;
    // Many partials per segment (waves well above segments): four waves per head.
    const bool wide = static_cast<int64_t>(a.waves) >= static_cast<int64_t>(kWideCombinePieces) * segs;
    const void* k = pick_combine(head_dim, dtype, wide);
    if (!k) return hipErrorInvalidValue;
    const unsigned ny = wide ? static_cast<unsigned>(a.group)
                             : static_cast<unsigned>((a.group + kBlockWaves - 1) / kBlockWaves);
    // Walk the workers' split-segment entries when they are fewer than the
    // segments (many short rows): each worker starts at most one split segment.
    DecodeArgs c = a;
    c.combine_by_worker = a.waves < segs ? 1 : 0;
    void* args[] = {&c};
    const dim3 grid = c.combine_by_worker
                          ? dim3(static_cast<unsigned>(a.waves / a.group_waves), ny * a.group_waves)
                          : dim3(static_cast<unsigned>(segs), ny);
    return launch_kernel(k, grid, dim3(kBlockThreads), args, 0, s, ev);
}

int decode_split_blocks_per_cu(int head_dim, int dtype, int batch) {
    const void* k = pick_split(head_dim, dtype, false, false);
    if (!k) return 0;
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k, kSplitBlockThreads, prefix_lds_bytes(batch)) !=
        hipSuccess)
        return 0;
    return n;
}

}  // namespace hck
