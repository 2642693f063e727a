// Host-side launchers for the library's HIP kernels (internal interface).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "hotcold_kv.h"

namespace hck {

// Page-table entry tags (KV_PAGE_COLD, KV_PAGE_STAGED) and the id below them.
constexpr int32_t kPageCold = KV_PAGE_COLD;
constexpr int32_t kPageStaged = KV_PAGE_STAGED;
constexpr int32_t kPageIdMask = KV_PAGE_STAGED - 1;

enum { kDtypeBf16 = 0, kDtypeF32 = 1 };

// Waves per 256-thread block of the decode kernel.
constexpr int kBlockWavesHost = 4;

// Where the pages of one pool live.  The slice of page p for layer l (its K
// and V tiles of every KV head, [kv_head][K tile, V tile]) starts at
// base + p * page_stride + l * layer_stride.  The hot pool is layer-major
// (page_stride = one slice, layer_stride = all of the pool's slices of one
// layer), so one layer's decode reads within 1 / num_layers of the pool; the
// cold pool is page-major (page_stride = one page, layer_stride = one slice),
// each 16-token block contiguous as the capacity tier stores it.
struct PoolGeom {
    char* base = nullptr;
    int64_t page_stride = 0;
    int64_t layer_stride = 0;
};
__host__ __device__ __forceinline__ char* slice_at(const PoolGeom& g, int64_t page, int64_t layer) {
    return g.base + page * g.page_stride + layer * g.layer_stride;
}

// Everything the split-K decode kernel and its combine read.
struct DecodeArgs {
    const char* hot;          // slice of hot page 0 for the decoded layer
    int64_t hot_stride;       // bytes between the slices of consecutive hot page ids
    int32_t num_pages;        // hot pages; ids outside [0, num_pages) are rejected
    int32_t num_kv_heads;
    int32_t group;            // query heads per KV head (1..16)
    int32_t num_q_heads;
    const void* q;            // [batch][num_q_heads][head_dim]
    const int32_t* page_table;
    int64_t pt_stride;
    const int32_t* seq_lens;  // [batch]
    int32_t batch;
    int32_t waves;            // number of waves the work is split over
    int32_t group_waves;      // waves sharing one work unit, one KV head each (1, or 4 = a block)
    float scale_log2;         // softmax scale * log2(e)
    float* part_o;            // [slots][group][head_dim] unnormalised partial outputs
    float* part_ml;           // [slots][2][group] running max (log2 domain) and weight sum
    int32_t* row_pref;        // [batch + 1] pages before each row (written by the split, read by the combine)
    int32_t* split_segs;      // [waves / group_waves] per worker, the segment (b * heads + head group)
                              // whose first piece it holds while later workers hold the rest, or -1
                              // (written by a separate-merge split, read by the combine)
    int32_t combine_by_worker;  // set by the combine launch: its grid walks split_segs, not all segments
    void* out;                // [batch][num_q_heads][head_dim]
    int32_t* counters;        // [batch * num_kv_heads] arrival counters, zero between calls
    int32_t fused;            // 1: the last wave of each (b, g) merges its partials
    // Tiered entries (honoured when `tiered` is set): KV_PAGE_COLD names a page
    // of the cold pool, KV_PAGE_STAGED a slot of this layer's staging buffer.
    int32_t tiered;
    const char* cold;         // slice of cold page 0 for the decoded layer (device-visible address)
    int64_t cold_stride;      // bytes between the slices of consecutive cold page ids
    int32_t num_cold_pages;
    const char* stage;        // staging buffer of this layer: [slot][kv_head][K tile, V tile]
    int32_t num_stage_slots;
    int64_t slice_bytes;      // bytes of one staging slot
    int32_t valu;             // 1: the split runs its products on the vector ALU (bf16, group <= 8)
    // Fused append (nullable): row b's token L - 1, [batch][num_kv_heads][head_dim], written
    // into its page before the page is read.
    const void* k_new;
    const void* v_new;
};

// Events a launch records at its kernel's start and end (the library's
// profiling); both null for a plain launch.  The timestamps come from the
// dispatch itself, so they bracket the kernel and nothing else.
struct LaunchEvents {
    hipEvent_t start = nullptr;
    hipEvent_t stop = nullptr;
};

inline hipError_t launch_kernel(const void* k, dim3 grid, dim3 block, void** args, size_t lds,
                                hipStream_t s, const LaunchEvents& ev) {
    if (ev.start && ev.stop) return hipExtLaunchKernel(k, grid, block, args, lds, s, ev.start, ev.stop, 0);
    return hipLaunchKernel(k, grid, block, args, lds, s);
}

// Waves that share one work unit of the decode split, one KV head each.  With
// four, a unit is one page of four KV heads and the four waves of a group read
// their heads' tiles of the same page side by side, which HBM serves faster
// than four unrelated pages (DRAM row locality).  Four when the KV heads come
// in fours and the waves in whole groups, else one (a unit is one page of one
// KV head).  The decode and its partition table follow the same rule.
#ifndef HCK_GROUP_WAVES
#define HCK_GROUP_WAVES 4
#endif
constexpr int kGroupWaves = HCK_GROUP_WAVES;
inline int decode_group_waves(int num_kv_heads, int waves) {
    return (num_kv_heads % kGroupWaves == 0 && waves % kGroupWaves == 0) ? kGroupWaves : 1;
}

// Bytes of partial results for `slots` slots.
inline size_t decode_partials_bytes(int64_t slots, int group, int head_dim) {
    return static_cast<size_t>(slots) * group * (head_dim + 2) * sizeof(float);
}

// Decode workspace: the partials, then the row page prefix (batch + 1 int32),
// then one split-segment entry per worker (at most `waves` int32), rounded up
// to 256 bytes.
inline size_t decode_workspace_bytes(int64_t slots, int group, int head_dim, int batch, int waves) {
    const size_t n = decode_partials_bytes(slots, group, head_dim) +
                     (static_cast<size_t>(batch) + 1 + static_cast<size_t>(waves)) * 4;
    return (n + 255) & ~static_cast<size_t>(255);
}

// The decode call behind paged_decode_attention and its no-allocation variant
// (host runtime).  With no_alloc the call takes no profiling events.
int decode_impl(kv_pool* pool, int32_t layer, const void* q, const int32_t* page_table, int64_t pt_stride,
                const int32_t* seq_lens, int32_t batch, int32_t num_q_heads, float scale, void* out,
                void* workspace, size_t ws_bytes, kv_stream_t stream, bool no_alloc,
                const void* k_new = nullptr, const void* v_new = nullptr);

// Device address of the no-allocation decode's scratch array on `device`
// (the current device); taken once per device and kept (noalloc.hip).
hipError_t scratch_address(int device, void** out);
// That address for a pool's device, taken when the pool was created
// (host runtime); KV_ERR_INVALID for a NULL or metadata-only pool.
int pool_scratch(kv_pool* pool, void** out);

hipError_t launch_decode_split(const DecodeArgs& a, int head_dim, int dtype, hipStream_t s,
                               const LaunchEvents& ev = {});
hipError_t launch_decode_combine(const DecodeArgs& a, int head_dim, int dtype, hipStream_t s,
                                 const LaunchEvents& ev = {});
// Largest batch the decode kernels accept (bounds the counter array).
constexpr int kMaxDecodeBatch = 8192;
// Resident 256-thread blocks per CU of the split kernel (0 if unsupported shape).
int decode_split_blocks_per_cu(int head_dim, int dtype, int batch);

// (waves + batch * num_kv_heads) records of 4 int32: (b, g, first page, end page).
hipError_t launch_gather_rows(const int32_t* pt, int64_t stride, int32_t max_sessions,
                              const int32_t* sids, int32_t n, int32_t* out, hipStream_t s);
hipError_t launch_partition(const int32_t* seq_lens, int batch, int num_kv_heads, int waves,
                            int group_waves, int64_t pt_stride, int32_t* slots, hipStream_t s);

struct CopyEntry {
    int32_t src;       // source page id, or -1: no copy
    int32_t dst;       // destination page id
    int32_t pt_index;  // page-table element to write, or -1
    int32_t pt_value;  // value written there
};

// For n entries (device array): copies `layers` slices of slice_bytes each
// (a multiple of 4 KiB), slice l of page e.src in `src` to slice l of page
// e.dst in `dst`, where e.src >= 0, and writes page_table[e.pt_index] =
// e.pt_value where e.pt_index >= 0.  Whole pages between the pools: layers =
// num_layers.  One layer's slices into the staging buffer: layers = 1, src
// based at that layer.  by_layer walks the copy layer by layer instead of page
// by page (for copies out of the layer-major hot pool).  max_blocks caps the
// persistent grid (0: the default).
hipError_t launch_page_copy(const PoolGeom& src, const PoolGeom& dst, int64_t slice_bytes, int32_t layers,
                            bool by_layer, const CopyEntry* entries, int32_t n, int32_t* page_table,
                            int32_t max_blocks, hipStream_t s, const LaunchEvents& ev = {});

hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t value, hipStream_t s);

// Streaming read of `bytes` (a multiple of 16) at buf by `blocks` blocks; one
// XOR word per block to out[0 .. blocks).
hipError_t launch_read_probe(const void* buf, int64_t bytes, uint32_t* out, int32_t blocks, hipStream_t s);

// page_table[e.pt_index] = e.pt_value for each of n entries with pt_index >= 0
// (no copies): the second phase of a promotion.
hipError_t launch_table_writes(const CopyEntry* entries, int32_t n, int32_t* page_table, hipStream_t s);

struct SynthArgs {
    PoolGeom hot;
    PoolGeom cold;       // for rows naming spilled pages (KV_PAGE_COLD)
    int64_t slice_bytes;
    const int32_t* row;  // device page-table row of the session
    int32_t first_page;  // first logical page filled
    int32_t num_pages;   // pages filled
    int32_t num_layers, num_kv_heads, head_dim, dtype;
    int32_t gen_sid;
    uint64_t seed;
    float value_mult;
};
hipError_t launch_fill_synthetic(const SynthArgs& a, hipStream_t s);

struct WriteArgs {
    PoolGeom hot;
    PoolGeom cold;       // for rows naming spilled pages (KV_PAGE_COLD)
    const int32_t* row;  // device page-table row of the session
    int32_t num_kv_heads, head_dim, dtype, layer;
    int32_t num_layers = 1;  // layers [layer, layer + num_layers)
    int32_t tok_begin, n_tok;
    const void* k;       // [num_layers][n_tok][num_kv_heads][head_dim]
    const void* v;
};
hipError_t launch_write_tokens(const WriteArgs& a, hipStream_t s);

// Where one appended token goes: its page (a hot id, or KV_PAGE_COLD | cold id
// for a spilled page) and its slot in the page.
struct AppendEntry {
    int32_t page;
    int32_t slot;
};

// Batches up to this many rows carry their entries in the kernel arguments
// (2 KiB), so a decode-step append needs no copy list and no staging slot.
constexpr int kAppendInline = 256;

struct AppendArgs {
    PoolGeom hot;
    PoolGeom cold;
    const AppendEntry* entries;  // device [n] when n > kAppendInline
    int32_t n;
    int32_t num_kv_heads, head_dim, dtype, layer;
    const void* k;               // [n][num_kv_heads][head_dim]
    const void* v;
    AppendEntry inline_entries[kAppendInline];  // the entries when n <= kAppendInline
};
hipError_t launch_append_tokens(const AppendArgs& a, hipStream_t s);

// Appends resolved on the device through a page table: entry r is token
// positions[r] of table row rows[r], for layers [layer, layer + num_layers).
struct AppendTableArgs {
    PoolGeom hot;
    PoolGeom cold;
    int32_t num_hot, num_cold;   // valid page ids of each pool
    const int32_t* table;        // device [table_rows][pt_stride]
    int64_t pt_stride;
    int32_t table_rows;
    const int32_t* rows;         // device [n]
    const int32_t* positions;    // device [n]
    int32_t n;
    int32_t num_kv_heads, head_dim, dtype, layer, num_layers;
    const void* k;               // [num_layers][n][num_kv_heads][head_dim]
    const void* v;
};
hipError_t launch_append_table(const AppendTableArgs& a, hipStream_t s);

}  // namespace hck
