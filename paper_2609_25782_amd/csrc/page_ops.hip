// Page movement and page-content kernels for gfx950.
//
//  - page_copy_kernel: whole-page copies between pools with an optional
//    page-table write per entry.  Resume (data path 2) gathers cold pages into
//    free hot pages and rewrites the sessions' rows in the same launch; eviction
//    (data path 4) scatters the pages that have no valid cold copy and clears
//    the rows, also in one launch.  The copy
//    is byte for byte, 16-byte vector loads and stores, several loads in
//    flight per thread before the first store.
//  - fill kernels for page tables and for synthetic page contents.
//  - write_tokens_kernel: fresh K/V into a session's hot pages (data path 3).
//  - partition kernels: the decode work split written out as a table.

#include "device_common.h"
#include "kernels.h"

namespace hck {
namespace {

#ifndef HCK_COPY_NONTEMPORAL
#define HCK_COPY_NONTEMPORAL 1
#endif
// Two launch shapes, chosen by the size of the copy (measured with 32 KiB and
// 1.5 MiB pages, destinations scattered over the hot pool):
//  - up to HCK_COPY_FINE_ROWS rows of 4 KiB (16 GiB): one 4 KiB row per block
//    iteration on a grid of up to HCK_COPY_FINE_BLOCKS blocks, i.e. one to a
//    few rows per block.  Small blocks that retire and are replaced keep every
//    CU busy to the end; the 1-layer resume of 345 MB runs 10% faster and
//    single 48-layer sessions of 6-13 GB 10-12% faster than with the coarse shape.
//  - larger copies: chunks of up to HCK_COPY_MAX_UNROLL rows on a persistent
//    grid of HCK_COPY_MAX_BLOCKS blocks (64 per CU on 256 CUs), which is 3%
//    faster for the 65 GB batched resume of 1.5 MiB pages.  A copy-block budget
//    set by the caller also takes this shape, with the budget as the grid.
#ifndef HCK_COPY_FINE_ROWS
#define HCK_COPY_FINE_ROWS (int64_t(4) << 20)
#endif
#ifndef HCK_COPY_FINE_BLOCKS
#define HCK_COPY_FINE_BLOCKS (int64_t(1) << 20)
#endif
#ifndef HCK_COPY_MAX_BLOCKS
#define HCK_COPY_MAX_BLOCKS 16384
#endif
#ifndef HCK_COPY_MAX_UNROLL
#define HCK_COPY_MAX_UNROLL 8
#endif

// The slice of layer `layer` of the page a session row names: a hot page, or a
// spilled page of the cold pool (KV_PAGE_COLD).  The host writes rows only
// with such entries.
__device__ __forceinline__ char* entry_slice(const PoolGeom& hot, const PoolGeom& cold, int32_t pid, int layer) {
    return (pid & kPageCold) ? slice_at(cold, pid & kPageIdMask, layer) : slice_at(hot, pid, layer);
}

// A block copies chunks of `U` x 4 KiB: every thread moves U 16-byte words, all
// loads issued before the first store.  The host picks U so that a chunk
// divides a slice (one layer of a page, a multiple of 4 KiB: two tiles of at
// least 2 KiB per KV head), so no chunk crosses from one slice to the next and
// the body has no bounds checks; each side maps (page, slice) through its own
// pool geometry.  The grid is persistent: block i takes chunks i, i + grid, ...
// of the whole copy list, so a multi-GB resume is a few thousand long-lived
// blocks rather than millions of short ones.  Chunks are walked page by page,
// or with `by_layer` layer by layer (every page's slice of layer 0 first): a
// copy out of the layer-major hot pool then reads within one layer's share of
// it at a time, which address translation serves far better than slices
// spread over the whole pool (reads stall on it; the scattered writes of the
// other direction are posted and hurt less).
template <int U>
__global__ __launch_bounds__(kBlockThreads) void page_copy_kernel(
    const PoolGeom src, const PoolGeom dst, const CopyEntry* __restrict__ entries, int32_t n,
    int chunks_per_entry, int chunks_per_slice, int by_layer, int32_t* __restrict__ page_table) {
    const int64_t total = static_cast<int64_t>(n) * chunks_per_entry;
    const int64_t per_layer = static_cast<int64_t>(n) * chunks_per_slice;
    for (int64_t flat = blockIdx.x; flat < total; flat += gridDim.x) {
        int ent, layer, cs;
        if (by_layer) {
            layer = static_cast<int>(flat / per_layer);
            const int64_t rem = flat % per_layer;
            ent = static_cast<int>(rem / chunks_per_slice);
            cs = static_cast<int>(rem % chunks_per_slice);
        } else {
            ent = static_cast<int>(flat / chunks_per_entry);
            const int chunk = static_cast<int>(flat % chunks_per_entry);
            layer = chunk / chunks_per_slice;
            cs = chunk % chunks_per_slice;
        }
        const CopyEntry e = entries[ent];
        if (layer == 0 && cs == 0 && threadIdx.x == 0 && e.pt_index >= 0) page_table[e.pt_index] = e.pt_value;
        if (e.src < 0) continue;
        const int64_t off = static_cast<int64_t>(cs) * U * kBlockThreads * 16;
        const u32x4* s = reinterpret_cast<const u32x4*>(slice_at(src, e.src, layer) + off) + threadIdx.x;
        u32x4* d = reinterpret_cast<u32x4*>(slice_at(dst, e.dst, layer) + off) + threadIdx.x;
        u32x4 buf[U];
#pragma unroll
        for (int i = 0; i < U; ++i)
            buf[i] = HCK_COPY_NONTEMPORAL ? __builtin_nontemporal_load(s + i * kBlockThreads)
                                          : s[i * kBlockThreads];
#pragma unroll
        for (int i = 0; i < U; ++i) {
            if (HCK_COPY_NONTEMPORAL)
                __builtin_nontemporal_store(buf[i], d + i * kBlockThreads);
            else
                d[i * kBlockThreads] = buf[i];
        }
    }
}

__global__ __launch_bounds__(kBlockThreads) void table_writes_kernel(const CopyEntry* __restrict__ entries,
                                                                     int32_t n, int32_t* page_table) {
    for (int32_t i = static_cast<int32_t>(blockIdx.x * kBlockThreads + threadIdx.x); i < n;
         i += static_cast<int32_t>(gridDim.x * kBlockThreads)) {
        const CopyEntry e = entries[i];
        if (e.pt_index >= 0) page_table[e.pt_index] = e.pt_value;
    }
}

// Streaming read of a whole buffer: each block reads whole chunks of 32 KiB
// (256 threads x 8 nontemporal 16-byte loads, all in flight together), chunks
// dealt to the blocks in turn, and folds them into an XOR, one word per block,
// so the loads cannot be dropped.  Contiguous chunks per block read faster
// than the same loads strided over the whole grid (DRAM row locality).  It
// measures the read rate the GPU reaches on plain sequential data with the
// loads the decode kernel uses.
__global__ __launch_bounds__(kBlockThreads) void read_probe_kernel(const u32x4* __restrict__ p, int64_t n16,
                                                                   uint32_t* __restrict__ out) {
    constexpr int U = 8;
    constexpr int64_t kChunk = static_cast<int64_t>(kBlockThreads) * U;  // 16-byte elements
    const int64_t nchunks = n16 / kChunk;
    u32x4 acc = {0u, 0u, 0u, 0u};
    for (int64_t c = blockIdx.x; c < nchunks; c += gridDim.x) {
        const u32x4* q = p + c * kChunk + threadIdx.x;
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(q + u * kBlockThreads);
#pragma unroll
        for (int u = 0; u < U; ++u) acc ^= v[u];
    }
    // elements past the last whole chunk
    for (int64_t i = nchunks * kChunk + static_cast<int64_t>(blockIdx.x) * kBlockThreads + threadIdx.x; i < n16;
         i += static_cast<int64_t>(gridDim.x) * kBlockThreads)
        acc ^= __builtin_nontemporal_load(p + i);
    unsigned x = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) x ^= __shfl_xor(x, o);
    __shared__ unsigned s_x[kBlockWaves];
    if ((threadIdx.x & (kWave - 1)) == 0) s_x[threadIdx.x / kWave] = x;
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned r = 0;
        for (int w = 0; w < kBlockWaves; ++w) r ^= s_x[w];
        out[blockIdx.x] = r;
    }
}

__global__ __launch_bounds__(kBlockThreads) void fill_i32_kernel(int32_t* p, int64_t n, int32_t v) {
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlockThreads + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * kBlockThreads)
        p[i] = v;
}

// SplitMix64 output function of x + golden ratio (Steele, Lea and Flood 2014).
__device__ __forceinline__ uint64_t splitmix_mix(uint64_t x) {
    uint64_t z = x + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__device__ __forceinline__ float synth_value(uint64_t key, uint64_t coord, float mult) {
    const uint64_t h = splitmix_mix(key ^ coord);
    const int s = static_cast<int>(h & 0xFFFF) + static_cast<int>((h >> 16) & 0xFFFF) +
                  static_cast<int>((h >> 32) & 0xFFFF) + static_cast<int>(h >> 48) - 131070;
    return static_cast<float>(s) * mult;
}

__device__ __forceinline__ uint64_t synth_coord(int kind, int sid, int layer, int head, int token,
                                                int dim) {
    return (static_cast<uint64_t>(kind) << 62) | (static_cast<uint64_t>(sid) << 42) |
           (static_cast<uint64_t>(layer) << 36) | (static_cast<uint64_t>(head) << 32) |
           (static_cast<uint64_t>(token) << 8) | static_cast<uint64_t>(dim);
}

__device__ __forceinline__ unsigned short bf16_rne(float f) {
    const unsigned b = __builtin_bit_cast(unsigned, f);
    return static_cast<unsigned short>((b + 0x7FFFu + ((b >> 16) & 1u)) >> 16);
}

// One thread per 16-byte group of a session's pages.
__global__ __launch_bounds__(kBlockThreads) void fill_synthetic_kernel(SynthArgs a) {
    const bool bf16 = a.dtype == kDtypeBf16;
    const int elt = bf16 ? 2 : 4;
    const int x = 16 / elt;
    const int64_t tile = static_cast<int64_t>(kPageTokens) * a.head_dim * elt;
    const int64_t groups_per_page = a.slice_bytes * a.num_layers / 16;
    const int64_t total = groups_per_page * a.num_pages;
    const uint64_t key = splitmix_mix(a.seed);
    for (int64_t gi = static_cast<int64_t>(blockIdx.x) * kBlockThreads + threadIdx.x; gi < total;
         gi += static_cast<int64_t>(gridDim.x) * kBlockThreads) {
        const int page_idx = a.first_page + static_cast<int>(gi / groups_per_page);
        const int64_t byte = (gi % groups_per_page) * 16;
        const int32_t pid = a.row[page_idx];
        const int64_t lh = byte / (2 * tile);
        const int layer = static_cast<int>(lh / a.num_kv_heads);
        const int head = static_cast<int>(lh % a.num_kv_heads);
        const int64_t in_lh = byte % (2 * tile);
        const int kind = static_cast<int>(in_lh / tile);
        const int e0 = static_cast<int>((in_lh % tile) / elt);  // first element of the group
        unsigned words[4];
        if (bf16) {
            unsigned short v[8];
            for (int j = 0; j < 8; ++j) {
                int t, d;
                if (kind == 0) {
                    t = (e0 / x) % kPageTokens;
                    d = (e0 / (x * kPageTokens)) * x + j;
                } else {
                    t = (e0 + j) % kPageTokens;
                    d = (e0 + j) / kPageTokens;
                }
                v[j] = bf16_rne(synth_value(
                    key, synth_coord(kind, a.gen_sid, layer, head, page_idx * kPageTokens + t, d),
                    a.value_mult));
            }
            for (int j = 0; j < 4; ++j) words[j] = v[2 * j] | (static_cast<unsigned>(v[2 * j + 1]) << 16);
        } else {
            for (int j = 0; j < 4; ++j) {
                int t, d;
                if (kind == 0) {
                    t = (e0 / x) % kPageTokens;
                    d = (e0 / (x * kPageTokens)) * x + j;
                } else {
                    t = (e0 + j) % kPageTokens;
                    d = (e0 + j) / kPageTokens;
                }
                words[j] = __builtin_bit_cast(
                    unsigned, synth_value(key,
                                          synth_coord(kind, a.gen_sid, layer, head,
                                                      page_idx * kPageTokens + t, d),
                                          a.value_mult));
            }
        }
        *reinterpret_cast<u32x4*>(entry_slice(a.hot, a.cold, pid, layer) + byte % a.slice_bytes) =
            u32x4{words[0], words[1], words[2], words[3]};
    }
}

// One thread per (token, KV head, 16-byte group of dims).
// One 16-byte group of dims (x elements) of one token's K and V into the
// (layer, KV head) slice `lh` of its page, token slot `slot`: K is a 16-byte
// store (the group is contiguous in the K tile); V, dims-major and
// token-minor, takes one element store per dim.
__device__ __forceinline__ void write_token_group(char* lh, int64_t tile, int slot, int cd, int x, int elt,
                                                  const char* ksrc, const char* vsrc) {
    *reinterpret_cast<u32x4*>(lh + (static_cast<int64_t>(cd) * kPageTokens + slot) * x * elt) =
        *reinterpret_cast<const u32x4*>(ksrc);
    char* vt = lh + tile;
    for (int j = 0; j < x; ++j) {
        const int64_t e = static_cast<int64_t>(cd * x + j) * kPageTokens + slot;
        if (elt == 2)
            *reinterpret_cast<unsigned short*>(vt + e * 2) = reinterpret_cast<const unsigned short*>(vsrc)[j];
        else
            *reinterpret_cast<unsigned*>(vt + e * 4) = reinterpret_cast<const unsigned*>(vsrc)[j];
    }
}

// Fresh KV is read once from its source and not read again until a later
// decode step, long after it has left the caches: its 16-byte loads and stores
// are nontemporal by default (HCK_WRITE_NONTEMPORAL).
#ifndef HCK_WRITE_NONTEMPORAL
#define HCK_WRITE_NONTEMPORAL 1
#endif
__device__ __forceinline__ u32x4 stream_load(const u32x4* p) {
    if (HCK_WRITE_NONTEMPORAL) return __builtin_nontemporal_load(p);
    return *p;
}
__device__ __forceinline__ void stream_store(u32x4* p, const u32x4& v) {
    if (HCK_WRITE_NONTEMPORAL)
        __builtin_nontemporal_store(v, p);
    else
        *p = v;
}

// Tokens [tok_begin, tok_begin + n_tok) of layers [layer, layer + num_layers):
// one block per (page, KV head, layer).  The page's tokens in the range are
// read from the source rows ([layer][token][kv_head][head_dim], each token's
// dims contiguous) into LDS with 16-byte loads, then written out in the tile
// layouts with 16-byte stores: K as groups of x dims, consecutive threads on
// consecutive tokens; V transposed to dims-major rows of 16 tokens.  Slots of
// the page outside the range keep their bytes: a V store that would cover one
// of them is done element by element instead.
template <typename T>
__global__ __launch_bounds__(kBlockThreads) void write_tokens_kernel(WriteArgs a) {
    constexpr int x = 16 / sizeof(T);            // elements per 16 bytes
    constexpr int kMaxD = 128;
    __shared__ __align__(16) T s_k[kPageTokens][kMaxD + x];
    __shared__ __align__(16) T s_v[kPageTokens][kMaxD + x];
    const int D = a.head_dim;
    const int groups = D / x;
    const int64_t tile = static_cast<int64_t>(kPageTokens) * D * sizeof(T);
    const int p0 = a.tok_begin / kPageTokens;
    const int page = p0 + static_cast<int>(blockIdx.x);
    const int head = static_cast<int>(blockIdx.y);
    const int layer = a.layer + static_cast<int>(blockIdx.z);
    const int64_t layer_src = static_cast<int64_t>(blockIdx.z) * a.n_tok * a.num_kv_heads * D;
    const int t_base = page * kPageTokens;
    const int s0 = max(a.tok_begin, t_base) - t_base;                       // first slot written
    const int s1 = min(a.tok_begin + a.n_tok, t_base + kPageTokens) - t_base;  // one past the last
    const int tid = threadIdx.x;
    for (int e = tid; e < kPageTokens * groups; e += kBlockThreads) {
        const int t = e / groups, cd = e % groups;
        if (t < s0 || t >= s1) continue;
        const int64_t src =
            layer_src + (static_cast<int64_t>(t_base + t - a.tok_begin) * a.num_kv_heads + head) * D + cd * x;
        *reinterpret_cast<u32x4*>(&s_k[t][cd * x]) =
            stream_load(reinterpret_cast<const u32x4*>(static_cast<const T*>(a.k) + src));
        *reinterpret_cast<u32x4*>(&s_v[t][cd * x]) =
            stream_load(reinterpret_cast<const u32x4*>(static_cast<const T*>(a.v) + src));
    }
    __syncthreads();
    char* lh = entry_slice(a.hot, a.cold, a.row[page], layer) + static_cast<int64_t>(head) * 2 * tile;
    // K tile: [group][token][x]
    for (int e = tid; e < groups * kPageTokens; e += kBlockThreads) {
        const int cd = e / kPageTokens, t = e % kPageTokens;
        if (t < s0 || t >= s1) continue;
        stream_store(reinterpret_cast<u32x4*>(lh + (static_cast<int64_t>(cd) * kPageTokens + t) * 16),
                     *reinterpret_cast<const u32x4*>(&s_k[t][cd * x]));
    }
    // V tile: [dim][token]; one 16-byte store covers x consecutive tokens of a dim
    constexpr int kChunks = kPageTokens / x;
    T* vt = reinterpret_cast<T*>(lh + tile);
    for (int e = tid; e < D * kChunks; e += kBlockThreads) {
        const int d = e / kChunks, c = e % kChunks;
        const int t0 = c * x;
        if (t0 + x <= s0 || t0 >= s1) continue;
        if (t0 >= s0 && t0 + x <= s1) {
            T w[x];
#pragma unroll
            for (int j = 0; j < x; ++j) w[j] = s_v[t0 + j][d];
            stream_store(reinterpret_cast<u32x4*>(vt + static_cast<int64_t>(d) * kPageTokens + t0),
                         *reinterpret_cast<const u32x4*>(w));
        } else {
            for (int j = 0; j < x; ++j)
                if (t0 + j >= s0 && t0 + j < s1) vt[static_cast<int64_t>(d) * kPageTokens + t0 + j] = s_v[t0 + j][d];
        }
    }
}

// Row r of the batch: one token into page e[r].page (a hot id, or a cold id
// tagged KV_PAGE_COLD) at slot e[r].slot; K and V rows [n][kv_heads][head_dim].
__global__ __launch_bounds__(kBlockThreads) void append_tokens_kernel(const AppendArgs a) {
    const int elt = a.dtype == kDtypeBf16 ? 2 : 4;
    const int x = 16 / elt;
    const int groups = a.head_dim / x;
    const int64_t tile = static_cast<int64_t>(kPageTokens) * a.head_dim * elt;
    const int64_t total = static_cast<int64_t>(a.n) * a.num_kv_heads * groups;
    for (int64_t gi = static_cast<int64_t>(blockIdx.x) * kBlockThreads + threadIdx.x; gi < total;
         gi += static_cast<int64_t>(gridDim.x) * kBlockThreads) {
        const int cd = static_cast<int>(gi % groups);
        const int head = static_cast<int>((gi / groups) % a.num_kv_heads);
        const int r = static_cast<int>(gi / (static_cast<int64_t>(groups) * a.num_kv_heads));
        const AppendEntry e = a.n <= kAppendInline ? a.inline_entries[r] : a.entries[r];
        char* lh = entry_slice(a.hot, a.cold, e.page, a.layer) + static_cast<int64_t>(head) * 2 * tile;
        const int64_t src = ((static_cast<int64_t>(r) * a.num_kv_heads + head) * a.head_dim + cd * x) * elt;
        write_token_group(lh, tile, e.slot, cd, x, elt, static_cast<const char*>(a.k) + src,
                          static_cast<const char*>(a.v) + src);
    }
}

// Appends whose page is resolved on the device: entry r writes token
// positions[r] of batch row rows[r] for layers [layer, layer + num_layers),
// into the page that row's page-table entry names (a hot page, or a spilled
// page of the cold pool), at slot positions[r] % 16.  One thread per (layer,
// entry, KV head, 16-byte group of dims).  An entry whose row, position or
// page-table entry does not name a page of either pool writes nothing.
__global__ __launch_bounds__(kBlockThreads) void append_table_kernel(const AppendTableArgs a) {
    const int elt = a.dtype == kDtypeBf16 ? 2 : 4;
    const int x = 16 / elt;
    const int groups = a.head_dim / x;
    const int64_t tile = static_cast<int64_t>(kPageTokens) * a.head_dim * elt;
    const int64_t per_layer = static_cast<int64_t>(a.n) * a.num_kv_heads * groups;
    const int64_t total = per_layer * a.num_layers;
    for (int64_t gi = static_cast<int64_t>(blockIdx.x) * kBlockThreads + threadIdx.x; gi < total;
         gi += static_cast<int64_t>(gridDim.x) * kBlockThreads) {
        const int li = static_cast<int>(gi / per_layer);
        const int64_t wi = gi % per_layer;
        const int cd = static_cast<int>(wi % groups);
        const int head = static_cast<int>((wi / groups) % a.num_kv_heads);
        const int r = static_cast<int>(wi / (static_cast<int64_t>(groups) * a.num_kv_heads));
        const int32_t row = a.rows[r], pos = a.positions[r];
        if (row < 0 || row >= a.table_rows || pos < 0 || pos / kPageTokens >= a.pt_stride) continue;
        const int32_t pid = a.table[static_cast<int64_t>(row) * a.pt_stride + pos / kPageTokens];
        const unsigned id = static_cast<unsigned>(pid) & static_cast<unsigned>(kPageIdMask);
        const unsigned tag = static_cast<unsigned>(pid) >> 29;   // 0 hot, 2 cold; others name no page
        if (!((tag == 0 && id < static_cast<unsigned>(a.num_hot)) ||
              (tag == 2 && id < static_cast<unsigned>(a.num_cold))))
            continue;
        char* lh = entry_slice(a.hot, a.cold, pid, a.layer + li) + static_cast<int64_t>(head) * 2 * tile;
        const int64_t src = (((static_cast<int64_t>(li) * a.n + r) * a.num_kv_heads + head) * a.head_dim + cd * x) * elt;
        write_token_group(lh, tile, pos % kPageTokens, cd, x, elt, static_cast<const char*>(a.k) + src,
                          static_cast<const char*>(a.v) + src);
    }
}

__global__ __launch_bounds__(kBlockThreads) void partition_holes_kernel(int32_t* slots, int64_t n) {
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlockThreads + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * kBlockThreads) {
        reinterpret_cast<int4*>(slots)[i] = make_int4(-1, -1, 0, 0);
    }
}

// Rows of the pool's page table for a batch of session ids; an id outside
// [0, max_sessions) gives a row of -1.  One thread per output entry.
__global__ __launch_bounds__(kBlockThreads) void gather_rows_kernel(const int32_t* pt, int64_t stride,
                                                                    int32_t max_sessions,
                                                                    const int32_t* sids, int32_t n,
                                                                    int32_t* out) {
    const int64_t total = static_cast<int64_t>(n) * stride;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlockThreads + threadIdx.x; i < total;
         i += static_cast<int64_t>(gridDim.x) * kBlockThreads) {
        const int64_t row = i / stride;
        const int32_t sid = sids[row];
        out[i] = (sid >= 0 && sid < max_sessions) ? pt[static_cast<int64_t>(sid) * stride + i % stride] : -1;
    }
}

// One thread per worker: enumerate its pieces exactly as the decode kernel
// does (here the lanes of a hardware wave work on different decode workers),
// and write the record of each of its `group_waves` waves.
__global__ __launch_bounds__(kBlockThreads) void partition_kernel(const int32_t* seq_lens, int batch,
                                                                  int num_kv_heads, int waves,
                                                                  int group_waves, int64_t stride,
                                                                  int32_t* slots) {
    extern __shared__ int32_t s_pref[];
    block_prefix_pages(seq_lens, batch, stride, s_pref);
    __syncthreads();
    const int heads = num_kv_heads / group_waves;
    const int workers = waves / group_waves;
    const int64_t total = static_cast<int64_t>(lds_uniform(s_pref + batch)) * heads;
    for (int k = blockIdx.x * kBlockThreads + threadIdx.x; k < workers; k += gridDim.x * kBlockThreads) {
        int64_t u, u1;
        wave_units(total, k, workers, u, u1);
        while (u < u1) {
            const Piece pc = piece_at<false>(s_pref, batch, heads, k, u, u1);
            if (pc.p1 <= pc.p0) break;  // cannot happen for a consistent prefix; never spin
            for (int w = 0; w < group_waves; ++w)
                reinterpret_cast<int4*>(slots)[static_cast<int64_t>(pc.slot) * group_waves + w] =
                    make_int4(pc.b, pc.g * group_waves + w, pc.p0, pc.p1);
            u += pc.p1 - pc.p0;
        }
    }
}

int grid_for(int64_t work, int cap) {
    const int64_t b = (work + kBlockThreads - 1) / kBlockThreads;
    return static_cast<int>(b < 1 ? 1 : (b > cap ? cap : b));
}

}  // namespace

hipError_t launch_page_copy(const PoolGeom& src, const PoolGeom& dst, int64_t slice_bytes, int32_t layers,
                            bool by_layer, const CopyEntry* entries, int32_t n, int32_t* page_table,
                            int32_t max_blocks, hipStream_t s, const LaunchEvents& ev) {
    if (n <= 0) return hipSuccess;
    constexpr int64_t kRow = static_cast<int64_t>(kBlockThreads) * 16;  // 4 KiB
    if (slice_bytes % kRow || slice_bytes <= 0 || layers < 1) return hipErrorInvalidValue;
    const int64_t rows = slice_bytes / kRow;  // per slice
    // a caller's budget (max_blocks) keeps few blocks: they take the large chunks
    const bool fine = max_blocks <= 0 && rows * layers * n <= HCK_COPY_FINE_ROWS;
    constexpr int kMaxU = HCK_COPY_MAX_UNROLL;
    const int u = fine ? 1
                : (kMaxU >= 8 && rows % 8 == 0) ? 8
                : (kMaxU >= 4 && rows % 4 == 0) ? 4
                : (kMaxU >= 2 && rows % 2 == 0) ? 2 : 1;
    const int cps = static_cast<int>(rows / u);
    const int cpe = cps * layers;
    const int64_t work = static_cast<int64_t>(cpe) * n;
    const int64_t cap = max_blocks > 0 ? max_blocks : fine ? HCK_COPY_FINE_BLOCKS : HCK_COPY_MAX_BLOCKS;
    const int64_t blocks = work < cap ? work : cap;
    const void* k = u == 8   ? reinterpret_cast<const void*>(&page_copy_kernel<8>)
                    : u == 4 ? reinterpret_cast<const void*>(&page_copy_kernel<4>)
                    : u == 2 ? reinterpret_cast<const void*>(&page_copy_kernel<2>)
                             : reinterpret_cast<const void*>(&page_copy_kernel<1>);
    int bl = by_layer ? 1 : 0;
    void* args[] = {const_cast<PoolGeom*>(&src), const_cast<PoolGeom*>(&dst), &entries, &n,
                    const_cast<int*>(&cpe), const_cast<int*>(&cps), &bl, &page_table};
    return launch_kernel(k, dim3(static_cast<unsigned>(blocks)), dim3(kBlockThreads), args, 0, s, ev);
}

hipError_t launch_table_writes(const CopyEntry* entries, int32_t n, int32_t* page_table, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(table_writes_kernel, dim3(grid_for(n, 1024)), dim3(kBlockThreads), 0, s, entries, n,
                       page_table);
    return hipGetLastError();
}

hipError_t launch_read_probe(const void* buf, int64_t bytes, uint32_t* out, int32_t blocks, hipStream_t s) {
    if (blocks <= 0 || bytes <= 0 || bytes % 16) return hipErrorInvalidValue;
    hipLaunchKernelGGL(read_probe_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kBlockThreads), 0, s,
                       static_cast<const u32x4*>(buf), bytes / 16, out);
    return hipGetLastError();
}

hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t value, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(fill_i32_kernel, dim3(grid_for(n, 4096)), dim3(kBlockThreads), 0, s, p, n, value);
    return hipGetLastError();
}

hipError_t launch_fill_synthetic(const SynthArgs& a, hipStream_t s) {
    const int64_t groups = a.slice_bytes * a.num_layers / 16 * a.num_pages;
    if (groups <= 0) return hipSuccess;
    hipLaunchKernelGGL(fill_synthetic_kernel, dim3(grid_for(groups, 16384)), dim3(kBlockThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_write_tokens(const WriteArgs& a, hipStream_t s) {
    if (a.n_tok <= 0) return hipSuccess;
    if (a.head_dim > 128 || a.head_dim % 16) return hipErrorInvalidValue;
    if (a.num_layers < 1 || a.num_layers > 65535) return hipErrorInvalidValue;
    const int pages = (a.tok_begin + a.n_tok - 1) / kPageTokens - a.tok_begin / kPageTokens + 1;
    const dim3 grid(static_cast<unsigned>(pages), static_cast<unsigned>(a.num_kv_heads),
                    static_cast<unsigned>(a.num_layers));
    if (a.dtype == kDtypeBf16)
        hipLaunchKernelGGL(write_tokens_kernel<unsigned short>, grid, dim3(kBlockThreads), 0, s, a);
    else
        hipLaunchKernelGGL(write_tokens_kernel<unsigned>, grid, dim3(kBlockThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_append_tokens(const AppendArgs& a, hipStream_t s) {
    const int x = a.dtype == kDtypeBf16 ? 8 : 4;
    const int64_t work = static_cast<int64_t>(a.n) * a.num_kv_heads * (a.head_dim / x);
    if (work <= 0) return hipSuccess;
    hipLaunchKernelGGL(append_tokens_kernel, dim3(grid_for(work, 16384)), dim3(kBlockThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_append_table(const AppendTableArgs& a, hipStream_t s) {
    const int x = a.dtype == kDtypeBf16 ? 8 : 4;
    const int64_t work = static_cast<int64_t>(a.n) * a.num_kv_heads * (a.head_dim / x) * a.num_layers;
    if (work <= 0) return hipSuccess;
    hipLaunchKernelGGL(append_table_kernel, dim3(grid_for(work, 16384)), dim3(kBlockThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_gather_rows(const int32_t* pt, int64_t stride, int32_t max_sessions,
                              const int32_t* sids, int32_t n, int32_t* out, hipStream_t s) {
    const int64_t total = static_cast<int64_t>(n) * stride;
    if (total <= 0) return hipSuccess;
    hipLaunchKernelGGL(gather_rows_kernel, dim3(grid_for(total, 4096)), dim3(kBlockThreads), 0, s, pt,
                       stride, max_sessions, sids, n, out);
    return hipGetLastError();
}

hipError_t launch_partition(const int32_t* seq_lens, int batch, int num_kv_heads, int waves,
                            int group_waves, int64_t pt_stride, int32_t* slots, hipStream_t s) {
    if (group_waves < 1 || num_kv_heads % group_waves || waves % group_waves) return hipErrorInvalidValue;
    const int64_t n = static_cast<int64_t>(waves) + static_cast<int64_t>(batch) * num_kv_heads;
    hipLaunchKernelGGL(partition_holes_kernel, dim3(grid_for(n, 4096)), dim3(kBlockThreads), 0, s, slots, n);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || batch == 0) return e;
    const size_t lds = static_cast<size_t>(batch + 1) * sizeof(int32_t);
    hipLaunchKernelGGL(partition_kernel, dim3(grid_for(waves / group_waves, 1024)), dim3(kBlockThreads), lds, s,
                       seq_lens, batch, num_kv_heads, waves, group_waves, pt_stride, slots);
    return hipGetLastError();
}

}  // namespace hck
