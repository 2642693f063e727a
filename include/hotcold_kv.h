/*
 * hotcold_kv.h — C ABI of the hot-cold KV-cache hot path for AMD Instinct MI355X (gfx950).
 *
 * The paper ("Hot-Cold Tiering of HBM and High Bandwidth Flash for Agentic LLM
 * Serving") splits the KV cache of agentic sessions into a hot set, the KV of
 * sessions that are decoding and that every decode step reads (Sec. I; Sec. II,
 * "Agentic AI Serving"), and a cold pool holding what paused sessions have
 * written, read only when a session resumes.  The hot set lives in the fast tier; the cold pool in
 * a capacity tier (Sec. III, first paragraph).  This library implements the
 * data-parallel part of that hierarchy on one GPU:
 *
 *   - decode attention over every active session's hot pages   (data path 1)
 *   - resume: gather a paused session's pages into free hot pages and
 *     rewrite its page table                                     (data path 2)
 *   - writing fresh KV into hot pages                            (data path 3)
 *   - eviction with write-on-evict                               (data path 4)
 *
 * (Data paths 1-4: Sec. III, "Architecture and data paths".)
 *
 * The cold tier is a second page pool in device memory standing in for the
 * flash tier, or, optionally, a pool in pinned host memory read over PCIe.
 *
 * ---------------------------------------------------------------------------
 * Page layout
 * ---------------------------------------------------------------------------
 * KV is stored in pages of KV_PAGE_TOKENS = 16 tokens (paged KV cache, Sec. II;
 * 16 tokens x 96 KiB per token = the paper's 1.5 MiB block, Sec. IV).  Hot and
 * cold pools have separate int32 page-id spaces.  One page holds, for every
 * layer and KV head, a K tile and a V tile:
 *
 *   page    = [num_layers][slice]        slice = [num_kv_heads][2 (K tile, V tile)][tile]
 *   tile    = KV_PAGE_TOKENS * head_dim elements
 *   K tile  : element (token t, dim d) at index ((d / x) * 16 + t) * x + d % x,
 *             x = 16 bytes / element size (8 for bf16, 4 for float32):
 *             16-byte groups of x consecutive dims, token-minor.
 *   V tile  : element (t, d) at index d * 16 + t (dims-major, token-minor).
 *
 * page_bytes = num_layers * slice_bytes, slice_bytes = num_kv_heads * 2 * 16 *
 * head_dim * element size (1.5 MiB pages and 32 KiB slices for 48 layers x 4
 * KV heads x 128 dims x bf16).
 *
 * Where the pages sit:
 *   cold pool  page-major: page c is contiguous at cold_base + c * page_bytes,
 *              in the order above (the capacity tier's 1.5 MiB block);
 *   hot pool   layer-major: the slice of page p for layer l is at
 *              hot_base + (l * num_hot_pages + p) * slice_bytes.
 * A decode step reads one layer of every active page; layer-major keeps those
 * reads within 1 / num_layers of the hot pool, which the GPU's address
 * translation serves with far fewer misses than the same slices spread over
 * the whole pool.  Copies between the pools convert one layout into the other.
 *
 * A page table is int32 [rows][stride]; row r, entry i is the hot page holding
 * tokens 16 i .. 16 i + 15 of that row's session, -1 when unused.
 *
 * ---------------------------------------------------------------------------
 * Conventions
 * ---------------------------------------------------------------------------
 *  - Every call returns a status code (KV_OK or a negative KV_ERR_*).  No C++
 *    exception crosses this boundary.  kv_last_error() gives a message for the
 *    calling thread's last failure.
 *  - All buffers are owned by the caller and must outlive the pool.  The
 *    library owns only host bookkeeping, a small pinned staging ring, a small
 *    device buffer for copy lists and a 512 KiB array of decode counters.
 *  - Device work is enqueued on the caller's stream (kv_stream_t is a
 *    hipStream_t; NULL is the default stream) and the call returns without
 *    waiting for it.  Asynchronous device faults surface at the caller's next
 *    synchronisation.
 *  - A failing call changes nothing: no bookkeeping, no page table, no pages.
 *  - A pool is externally synchronised: one thread at a time.  Work on one
 *    stream is ordered; across streams the caller orders it with events, with
 *    one exception the pool handles itself: hot pages freed by an eviction or
 *    a destroy are not handed out to a call on another stream before the
 *    freeing call's device work has finished, on whichever streams the
 *    freeing calls ran.  Other readers of a session's pages (a decode, a
 *    resume still copying, on another stream) are the caller's to order
 *    before the call that frees those pages, hot or cold.
 */
#ifndef HOTCOLD_KV_H
#define HOTCOLD_KV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KV_PAGE_TOKENS 16

enum kv_status {
    KV_OK = 0,
    KV_ERR_INVALID = -1,        /* bad argument, descriptor, id or size */
    KV_ERR_STATE = -2,          /* session in the wrong state for the call */
    KV_ERR_NO_HOT_PAGES = -3,   /* hot pool has too few free pages */
    KV_ERR_NO_COLD_PAGES = -4,  /* cold pool has too few free pages */
    KV_ERR_HIP = -5,            /* a HIP runtime call failed (message has detail) */
    KV_ERR_OOM = -6             /* the library's own small allocations failed */
};

enum kv_dtype { KV_DTYPE_BF16 = 0, KV_DTYPE_F32 = 1 };

enum kv_cold_location {
    KV_COLD_DEVICE = 0,         /* cold pool in device memory (stands in for flash) */
    KV_COLD_PINNED_HOST = 1     /* cold pool in pinned host memory, read over PCIe */
};

enum kv_session_state { KV_SESSION_FREE = 0, KV_SESSION_ACTIVE = 1, KV_SESSION_PAUSED = 2 };

/* kv_pool_desc.flags */
#define KV_POOL_METADATA_ONLY 1  /* bookkeeping only: no buffers, no device work */

/*
 * Page-table entry tags.  An entry below KV_PAGE_STAGED is a hot page id;
 * KV_PAGE_COLD | c names page c of the cold pool (a spilled page, read by
 * decode in place); KV_PAGE_STAGED | s names slot s of the staging buffer of
 * the layer being decoded (see paged_decode_stage).  -1 and other negative
 * values are "no page".  Tagged entries are read only by pools with spill
 * enabled or a staging buffer set; elsewhere they are invalid ids.
 */
#define KV_PAGE_COLD (1 << 30)
#define KV_PAGE_STAGED (1 << 29)

/* Kernel ids for the profiling hook. */
enum kv_kernel_id {
    KV_KERNEL_DECODE_SPLIT = 0,   /* split-K paged decode attention */
    KV_KERNEL_DECODE_COMBINE = 1, /* combine of split partials */
    KV_KERNEL_PAGE_COPY = 2,      /* resume gather (cold -> hot) */
    KV_KERNEL_EVICT_COPY = 3,     /* eviction scatter and row clears (hot -> cold) */
    KV_KERNEL_PREFETCH_COPY = 4,  /* one layer's slices of spilled pages -> staging */
    KV_KERNEL_COUNT = 5
};

typedef void* kv_stream_t;
typedef struct kv_pool kv_pool;

typedef struct kv_pool_desc {
    int32_t num_layers;            /* >= 1 */
    int32_t num_kv_heads;          /* 1 .. 16 */
    int32_t head_dim;              /* 64 or 128 */
    int32_t page_size;             /* must be KV_PAGE_TOKENS */
    int32_t dtype;                 /* enum kv_dtype */
    int32_t num_hot_pages;         /* >= 0 */
    int32_t num_cold_pages;        /* >= 0 */
    int32_t cold_location;         /* enum kv_cold_location */
    int32_t max_sessions;          /* rows of the pool's page table */
    int32_t max_pages_per_session; /* row stride of the pool's page table */
    int32_t device;                /* HIP device ordinal holding the pools */
    int32_t flags;                 /* KV_POOL_METADATA_ONLY or 0 */
} kv_pool_desc;

typedef struct kv_pool_stats_t {
    int32_t free_hot_pages;
    int32_t free_cold_pages;
    int32_t active_sessions;
    int32_t paused_sessions;
    int64_t pages_to_cold;   /* pages written to the cold tier (write-on-evict) */
    int64_t pages_to_hot;    /* pages copied cold -> hot by resumes */
    int64_t bytes_to_cold;
    int64_t bytes_to_hot;
    int64_t resumes;         /* sessions resumed */
    int64_t evicts;          /* sessions evicted */
    int64_t resume_pages_resident; /* pages already in the hot tier when their session resumed */
    int64_t resume_pages_total;    /* pages of resumed sessions (hit rate = resident / total) */
    int64_t lru_evicted_pages;     /* pages of paused sessions evicted page by page (LRU) */
    int64_t spilled_pages;         /* pages placed or left in the cold tier by spill */
    int64_t promoted_pages;        /* spilled pages moved back to the hot tier */
    int64_t cold_active_pages;     /* now: pages of ACTIVE sessions living in the cold tier */
} kv_pool_stats_t;

/* ----------------------------------------------------------------------- */
/* Pool                                                                     */
/* ----------------------------------------------------------------------- */

/* Bytes of one page for this descriptor's layout (0 if the descriptor is invalid). */
size_t kv_page_bytes(const kv_pool_desc* desc);

/*
 * Create a pool over caller-owned memory.
 *   hot_base/hot_bytes   device memory, >= num_hot_pages * page_bytes, 256-byte aligned
 *   cold_base/cold_bytes device memory (KV_COLD_DEVICE) or pinned host memory
 *                        (KV_COLD_PINNED_HOST), >= num_cold_pages * page_bytes
 *   page_table           device int32 [max_sessions][max_pages_per_session]; the pool
 *                        fills it with -1 on `stream` and owns its contents afterwards
 * With KV_POOL_METADATA_ONLY all pointers may be NULL and no device is touched.
 * Hot and cold pages are handed out lowest id first (the paper leaves the
 * choice open; lowest-first makes page tables predictable).
 * Errors: KV_ERR_INVALID (descriptor or sizes), KV_ERR_HIP, KV_ERR_OOM.
 */
int kv_pool_create(const kv_pool_desc* desc, void* hot_base, size_t hot_bytes, void* cold_base,
                   size_t cold_bytes, int32_t* page_table, kv_stream_t stream, kv_pool** out);

/* Free host bookkeeping.  The caller must have synchronised streams using the pool. */
void kv_pool_destroy(kv_pool* pool);

/*
 * Introspection: free pages, sessions by state, pages and bytes copied in each
 * direction, resume hit-rate counts (resident / total pages of resumed
 * sessions, Sec. IV "Methodology"), LRU, spill and promotion counts.  *out is a
 * host struct the caller owns.  Errors: KV_ERR_INVALID (NULL argument).
 */
int kv_pool_stats(const kv_pool* pool, kv_pool_stats_t* out);

/* ----------------------------------------------------------------------- */
/* Sessions                                                                 */
/* ----------------------------------------------------------------------- */

/*
 * Create an ACTIVE session of seq_len tokens (a stand-in for prefill, which is
 * outside this library): allocates ceil(seq_len / 16) hot pages and writes the
 * session's page-table row.  hot_pages (host array, nullable) picks the exact
 * pages, which must be free and distinct.  NULL takes the lowest free ones; if
 * too few are free, least-recently-used pages of paused sessions are evicted
 * first (see kv_session_pause).  The page contents are left as they are: fill
 * them with kv_write_tokens or kv_fill_synthetic.  The new session id (lowest
 * free row) goes to *sid_out.
 * Errors: KV_ERR_INVALID, KV_ERR_NO_HOT_PAGES, KV_ERR_NO_COLD_PAGES (no room
 * for the cold copies of the pages that would have to be evicted).
 */
int kv_session_create(kv_pool* pool, int32_t seq_len, const int32_t* hot_pages,
                      kv_stream_t stream, int32_t* sid_out);

/*
 * Grow an ACTIVE session to new_seq_len tokens: decoding appends each new
 * token's KV (Sec. II; fresh KV goes to the fast tier, data path 3).  Pages for
 * the new tokens are allocated like kv_session_create's and appended to the
 * row; write the tokens' K and V with kv_write_tokens, kv_append_tokens or
 * kv_append_tokens_table.  The new tokens go into the partially filled tail
 * page first, so extending counts as writing that page: its cold copy is
 * dropped (the next eviction writes it again, Sec. III write-on-evict).
 * Errors: KV_ERR_INVALID (shrinking, row stride), KV_ERR_STATE (not ACTIVE, or
 * a spilled tail page shared with another session), KV_ERR_NO_HOT_PAGES,
 * KV_ERR_NO_COLD_PAGES.
 */
int kv_session_extend(kv_pool* pool, int32_t sid, int32_t new_seq_len, kv_stream_t stream);

/*
 * Pause an ACTIVE session (the agent waits for a tool or a user, Sec. II): no
 * data moves.  Its pages stay in the hot tier but become evictable, least
 * recently used first: the paper evicts LRU blocks, and since active blocks are
 * read every step, the oldest paused sessions' blocks go first (Sec. III,
 * "Eviction, resume and decode").  Pages of one session go in logical order.
 * Errors: KV_ERR_STATE (not ACTIVE).
 */
int kv_session_pause(kv_pool* pool, int32_t sid);

/*
 * Evict up to n least-recently-used resident pages of paused sessions to the
 * cold tier (write-on-evict: pages with a valid cold copy cost no write) and
 * free them; *evicted (nullable) gets the number evicted.
 * Errors: KV_ERR_NO_COLD_PAGES (nothing changes).
 */
int kv_evict_pages(kv_pool* pool, int32_t n, kv_stream_t stream, int32_t* evicted);

/*
 * Spill (enable = 1; off by default).  The paper does not pin active KV in HBM:
 * if HBM cannot hold even the decoding sessions' KV, blocks move to the
 * capacity tier instead of the call failing (Sec. III, "Eviction, resume and decode").  With
 * spill on, an allocating call that finds too few hot pages even after
 * evicting every resident page of paused sessions places the remaining new
 * pages in fresh cold pages (kv_session_create, kv_session_extend; hot pages
 * first in logical order), and a resume leaves the pages it cannot fetch in
 * the cold tier.  Such a page's row entry is KV_PAGE_COLD | cold id; decode
 * reads it from the cold tier, and kv_write_tokens / kv_fill_synthetic_pages
 * write it in place (refused with KV_ERR_STATE if that cold page is shared
 * with another session).  It is its own cold copy, so evicting it writes
 * nothing; its entry keeps naming the cold page until the page is fetched or
 * the whole session is evicted.
 * Errors: KV_ERR_INVALID; KV_ERR_STATE when turning spill off while some
 * session's row still names spilled pages (decode without spill would read
 * those entries as invalid ids): promote them or evict the session first.
 */
int kv_pool_set_spill(kv_pool* pool, int32_t enable);

/*
 * Move up to n spilled pages of ACTIVE sessions (session id order, logical page
 * order) back into hot pages, evicting resident pages of paused sessions by LRU
 * when no hot page is free: active pages are the more recently used (Sec.
 * III).  Their cold copies stay valid.  *promoted (nullable) gets the number
 * moved; it is smaller than n when the hot tier is full of active pages.
 * The row entries are rewritten on `stream` only after the copies, so a decode
 * of the same sessions on another stream may run meanwhile: it reads each page
 * either from its (unchanged) cold copy or from the finished hot copy.  The
 * LRU victims evicted to make room are pages of paused sessions, which decode
 * does not read.  Writes to those sessions on another stream
 * (kv_append_tokens, kv_write_tokens) are another matter: the caller orders
 * them around this call's work, since the copy could miss a write enqueued
 * before it and overwrite one enqueued after it.
 * Errors: KV_ERR_INVALID, KV_ERR_NO_COLD_PAGES (evicted pages need cold copies;
 * nothing changes).
 */
int kv_promote_pages(kv_pool* pool, int32_t n, kv_stream_t stream, int32_t* promoted);

/*
 * Lazy resume (spill on): the PAUSED sessions become ACTIVE without any copy;
 * their non-resident pages stay in the cold tier, named by KV_PAGE_COLD
 * entries, and decode reads them in place until kv_promote_pages moves them.
 * The paper fetches before decoding (Sec. III); with a cold tier as fast as
 * HBM this spreads the fetch over later steps under the caller's copy budget
 * instead of stalling the step that resumes.  Rows are rewritten on `stream`.
 * Errors: KV_ERR_INVALID (spill off, bad or duplicate ids), KV_ERR_STATE.
 */
int kv_resume_sessions_lazy(kv_pool* pool, const int32_t* sids, int32_t n, kv_stream_t stream);

/*
 * Register a PAUSED session of seq_len tokens whose KV already sits in the given
 * cold pages (host array of ceil(seq_len / 16) distinct ids).  Cold pages may be
 * shared with other paused sessions: KV never changes once written (Sec. II), so
 * a virtualised cold pool may alias them; they are reference counted.
 * Errors: KV_ERR_INVALID.
 */
int kv_session_import_cold(kv_pool* pool, int32_t seq_len, const int32_t* cold_pages,
                           int32_t* sid_out);

/* Release a session: its hot pages return to the free set (see the cross-stream
 * rule above), its cold references are dropped and its row is reset to -1. */
int kv_session_destroy(kv_pool* pool, int32_t sid, kv_stream_t stream);

/*
 * Describe a session.  Host outputs (any may be NULL): state, seq_len, and up to
 * `cap` entries each of its hot page ids (logical page order, -1 where the page
 * is not resident) and cold page ids (-1 where the page has no valid cold copy).
 */
int kv_session_info(const kv_pool* pool, int32_t sid, int32_t* state, int32_t* seq_len,
                    int32_t* hot_pages, int32_t* cold_pages, int32_t cap);

/*
 * Fresh KV into the hot tier (data path 3, Sec. III): write tokens
 * [tok_begin, tok_begin + n_tok) of an ACTIVE session for one layer.  k and v
 * are device arrays [n_tok][num_kv_heads][head_dim] of the pool's dtype.  Pages
 * written to lose their cold copy, so the next eviction writes them again.
 * On a KV_POOL_METADATA_ONLY pool only that bookkeeping happens (k and v are
 * ignored and may be NULL): a replay records appended tokens this way.
 * Errors: KV_ERR_INVALID (range beyond seq_len, bad layer), KV_ERR_STATE.
 */
int kv_write_tokens(kv_pool* pool, int32_t sid, int32_t layer, int32_t tok_begin, int32_t n_tok,
                    const void* k, const void* v, kv_stream_t stream);

/*
 * kv_write_tokens for layers [layer_begin, layer_begin + num_layers) in one
 * launch: k and v are device arrays [num_layers][n_tok][num_kv_heads][head_dim]
 * (16-byte aligned).  For writing a whole prompt's KV at once (a turn's tool
 * output or user text prefilled elsewhere), where one launch per layer would
 * spend more time launching than moving bytes.
 * Errors: KV_ERR_INVALID (layer range, token range, alignment), KV_ERR_STATE.
 */
int kv_write_tokens_layers(kv_pool* pool, int32_t sid, int32_t layer_begin, int32_t num_layers,
                           int32_t tok_begin, int32_t n_tok, const void* k, const void* v,
                           kv_stream_t stream);

/*
 * Batched append for a decode step (data path 3, Sec. III): for one layer, row
 * i of k and v (device arrays [n][num_kv_heads][head_dim], pool dtype) is
 * token positions[i] of ACTIVE session sids[i] (host arrays, n <= 8192).  One
 * launch writes every row.  Call kv_session_extend first so the positions lie
 * inside the sessions.  A token on a spilled page is written to its cold page
 * in place; hot pages written to lose their cold copy, as with kv_write_tokens.
 * All rows are checked before anything is written or launched.  On a
 * KV_POOL_METADATA_ONLY pool only the bookkeeping happens.
 * Errors: KV_ERR_INVALID (bad layer, a position outside its session, the same
 * token twice), KV_ERR_STATE (a session not ACTIVE, a spilled page shared with
 * another session).
 */
int kv_append_tokens(kv_pool* pool, int32_t layer, const int32_t* sids, const int32_t* positions, int32_t n,
                     const void* k, const void* v, kv_stream_t stream);

/*
 * A decode step's append resolved on the device (data path 3, Sec. III), so
 * that a whole serving step (append and decode for every layer) can be
 * captured into one HIP graph and replayed: no host bookkeeping, no copy list,
 * one kernel launch.  Entry i writes token positions[i] of row rows[i] of
 * `table` (device int32 [table_rows][pt_stride], e.g. a batch table from
 * paged_decode_gather_table, or the pool's own table) for layers
 * [layer_begin, layer_begin + num_layers): the page is the one that row's
 * entry positions[i] / 16 names (a hot page, or KV_PAGE_COLD | id: a spilled
 * page written in place) and the slot is positions[i] % 16.  rows and
 * positions are device int32 [n] (n <= 8192) read when the kernel runs, so a
 * graph replay takes their current values; k and v are device arrays
 * [num_layers][n][num_kv_heads][head_dim] of the pool's dtype, 16-byte aligned.
 * An entry whose row or position lies outside the table, or whose table entry
 * names no page of either pool (-1, a staged slot, an id out of range), writes
 * nothing.  Two entries naming the same token race.
 * The pool's bookkeeping is not read or changed.  Write-on-evict stays exact
 * for tokens that extend a session (positions at or past its length before its
 * last kv_session_extend): the extension already dropped the cold copy of the
 * page the new tokens go into.  Rewriting older tokens this way would leave
 * that page's cold copy stale; use kv_write_tokens for those.
 * Errors: KV_ERR_INVALID (layer range, n, NULL or misaligned buffers, table
 * shape, metadata-only pool), KV_ERR_HIP.
 */
int kv_append_tokens_table(kv_pool* pool, int32_t layer_begin, int32_t num_layers, const int32_t* table,
                           int64_t pt_stride, int32_t table_rows, const int32_t* rows,
                           const int32_t* positions, int32_t n, const void* k, const void* v,
                           kv_stream_t stream);

/*
 * Test and benchmark input: fill every slot of an ACTIVE session's pages, all
 * layers, with counter-based pseudo-normal values.  Element (kind, layer, head,
 * token, dim) of logical session gen_sid gets value(seed, coordinate) computed
 * with SplitMix64 (Steele, Lea and Flood 2014): h = mix(mix(seed) ^ c) with c
 * the packed coordinate (kind:2 | gen_sid:20 | layer:6 | head:5 | token:23 |
 * dim:8, kind 0 = K, 1 = V); s = sum of the four 16-bit fields of h - 131070;
 * value = float32(s) * value_mult, then rounded to bf16 (nearest-even) for bf16
 * pools.  Pages lose their cold copy.
 */
int kv_fill_synthetic(kv_pool* pool, int32_t sid, int32_t gen_sid, uint64_t seed,
                      float value_mult, kv_stream_t stream);

/*
 * kv_fill_synthetic restricted to logical pages [first_page, first_page +
 * num_pages) of the session (every slot of each, whatever seq_len is); only
 * those pages lose their cold copy.  A page holds the same values however
 * often it is filled, so appending tokens can refill the tail page.
 * Errors: KV_ERR_INVALID (range outside the session's pages), KV_ERR_STATE.
 */
int kv_fill_synthetic_pages(kv_pool* pool, int32_t sid, int32_t gen_sid, uint64_t seed,
                            float value_mult, int32_t first_page, int32_t num_pages,
                            kv_stream_t stream);

/*
 * Evict an ACTIVE session to the cold tier (data path 4) with write-on-evict
 * (Sec. III, "Memory hierarchy and write policy"): only pages without a valid
 * cold copy are copied, each into the lowest free cold page; pages that already
 * have one cost no write, so an unmodified page reaches the cold tier at most
 * once.  Then the session's hot pages are freed and its row set to -1; the
 * session becomes PAUSED.
 * Errors: KV_ERR_STATE (not ACTIVE), KV_ERR_NO_COLD_PAGES (nothing changes).
 */
int kv_evict_session(kv_pool* pool, int32_t sid, kv_stream_t stream);

/* Batched eviction: sessions in argument order, atomic as a whole, one launch
 * for all copies and row clears.  Errors as kv_evict_session. */
int kv_evict_sessions(kv_pool* pool, const int32_t* sids, int32_t n, kv_stream_t stream);

/*
 * Resume a PAUSED session (data path 2; Sec. III, "Eviction, resume and
 * decode": the KV is brought back into the fast tier before the session runs).
 * Only pages that are not resident are fetched: they get free hot pages (lowest
 * ids first, in logical page order; least-recently-used pages of other paused
 * sessions are evicted first if too few are free) and are copied cold -> hot
 * byte for byte.  The whole page-table row is written.  The cold copies stay
 * valid.  The statistics count resident and total pages (the resume hit rate).
 * Errors: KV_ERR_STATE (not PAUSED), KV_ERR_NO_HOT_PAGES, KV_ERR_NO_COLD_PAGES
 * (nothing changes).
 */
int kv_resume_session(kv_pool* pool, int32_t sid, kv_stream_t stream);

/* Batched resume: sessions in argument order, atomic as a whole, one launch. */
int kv_resume_sessions(kv_pool* pool, const int32_t* sids, int32_t n, kv_stream_t stream);

/*
 * Bandwidth budget of the page copies (resume, eviction): at most `blocks`
 * 256-thread blocks copy at once (0: the default, enough to fill the GPU).
 * It applies to the copy kernel only: pinned-host tier copies made by the DMA
 * engines (kv_pool_set_host_copy) do not use it.
 * The paper overlaps eviction and resume with decode (Sec. III, "Architecture
 * and data paths"); with a device-memory cold tier both share HBM, so a smaller
 * budget leaves decode more bandwidth and CU slots at the cost of a slower
 * resume.
 */
int kv_pool_set_copy_blocks(kv_pool* pool, int32_t blocks);

enum kv_host_copy {
    KV_HOST_COPY_DMA = 0,    /* the GPU's DMA engines, one copy per run of consecutive pages
                                (default) */
    KV_HOST_COPY_KERNEL = 1  /* the page-copy kernel reading or writing host memory over PCIe */
};
/*
 * How whole-page copies between a pinned-host cold pool and the hot pool
 * (resume, eviction, promotion) are done.  Both reach PCIe bandwidth alone
 * (the kernel somewhat more when pages are scattered), but copy waves waiting
 * on PCIe hold the CUs' memory pipelines and slow a decode running meanwhile
 * on another stream many times over, while the DMA engines use no CU.  The
 * one-layer gathers of paged_decode_prefetch always use the kernel.  No effect
 * on a device-memory cold pool.  KV_ERR_INVALID for other modes.
 */
int kv_pool_set_host_copy(kv_pool* pool, int32_t mode);

/* ----------------------------------------------------------------------- */
/* Streams on a share of the compute units                                  */
/* ----------------------------------------------------------------------- */

/*
 * The paper keeps fetches from the cold tier off the decode's path, running
 * beside it (Sec. III, "Architecture and data paths").  On one GPU a resume
 * copy and a decode launched on two plain streams share every CU: copy waves
 * then sit beside split waves, and the split, whose static partition waits
 * for its slowest wave, slows about threefold even when the copy's grid is
 * capped (kv_pool_set_copy_blocks).  Streams confined to disjoint sets of CUs
 * keep the two apart, so that only HBM bandwidth is shared.
 *
 * A "slot" is one CU of every XCD: the device has `xcds` XCDs of `slots` CUs
 * each, and slot j of XCD x is bit x + xcds * j of the HIP stream CU mask (the
 * driver spreads consecutive mask bits over the XCDs first, then over each
 * XCD's shader engines).  A range of slots therefore gives every XCD, and so
 * every L2, the same number of CUs.
 *
 * kv_device_cu_slots: the device's XCD count and CUs per XCD.
 * kv_stream_create_cu_slots: a new stream on `device` whose kernels run only
 *   on slots [slot_begin, slot_end) (0 <= begin < end <= slots).  The caller
 *   owns the stream and releases it with kv_stream_destroy after its work is
 *   done.  The decode's default grid (paged_decode_waves) has one block per CU
 *   on 192 CUs; on a stream with fewer CUs, set at most four waves per CU
 *   (kv_pool_set_decode_waves), or the split runs in two rounds.
 * KV_ERR_INVALID for a bad device, range or output pointer; KV_ERR_HIP when
 * the runtime refuses.
 */
int kv_device_cu_slots(int32_t device, int32_t* xcds, int32_t* slots);
int kv_stream_create_cu_slots(int32_t device, int32_t slot_begin, int32_t slot_end, kv_stream_t* stream_out);
int kv_stream_destroy(kv_stream_t stream);

/* ----------------------------------------------------------------------- */
/* Decode attention (data path 1)                                           */
/* ----------------------------------------------------------------------- */

/*
 * Number of waves the decode kernel splits the work over for this pool
 * (a persistent grid sized to the GPU), or the value set below.
 */
int32_t paged_decode_waves(const kv_pool* pool);

/*
 * Override the number of decode waves (>= 1); 0 restores the automatic choice.
 * A count that is not a multiple of 4 (or a pool whose KV heads are not) makes
 * every wave its own worker instead of four waves sharing each page (see
 * paged_decode_partition).
 */
int kv_pool_set_decode_waves(kv_pool* pool, int32_t waves);

enum kv_combine_mode {
    KV_COMBINE_SEPARATE = 0, /* partials merged by a second kernel (default) */
    KV_COMBINE_FUSED = 1     /* the last wave of each (row, KV head) merges them; every
                                wave's arrival is a device-scope release, which on gfx950
                                writes back its L2, and this mode is slower */
};
/* How paged_decode_attention merges its split partials.  The two modes merge
 * in different orders, so their results agree to float32 rounding, not bit for
 * bit; each mode on its own is deterministic. */
int kv_pool_set_decode_combine(kv_pool* pool, int32_t mode);

enum kv_decode_compute {
    KV_DECODE_MATRIX = 0, /* both products on the matrix cores (default) */
    KV_DECODE_VECTOR = 1  /* both products as bf16 dot2 on the vector ALU, with the same work
                             split, page loads and partial format; bf16 pools, at most 8 query
                             heads per KV head, separate merge only */
};
/* Which units the decode split kernel computes on.  The vector form exists to
 * measure the matrix-core choice; the two sum in different orders, so their
 * results agree to float32 rounding, not bit for bit.  Decode calls that the
 * vector form cannot serve return KV_ERR_INVALID. */
int kv_pool_set_decode_compute(kv_pool* pool, int32_t mode);

/*
 * The page table of a decode batch: row i of `table` (device int32
 * [n][max_pages_per_session]) becomes the pool's row for session sids[i]
 * (device int32 [n]), read on `stream`; an id outside [0, max_sessions) gives
 * a row of -1.  One launch per step serves every layer's paged_decode_attention
 * over the sessions decoding, with pt_stride = max_pages_per_session.
 * Errors: KV_ERR_INVALID (n < 0 or above 8192, NULL arrays).
 */
int paged_decode_gather_table(kv_pool* pool, const int32_t* sids, int32_t n, int32_t* table,
                              kv_stream_t stream);

/*
 * One-step-ahead prefetch of spilled pages (Sec. III: decode knows which
 * blocks it reads next and fetches them a step early).  Decode runs layer by
 * layer, so the step here is a layer: while layer l is decoded, the slices of
 * layer l + 1 of the batch's spilled pages are gathered from the cold tier into
 * HBM, and layer l + 1 then reads only HBM.
 *
 * Whether staging pays depends on the cold tier and on the share of spilled
 * pages.  Over device memory it only adds an HBM write and read per spilled
 * byte.  Over PCIe it pays when one layer's spilled slices cross PCIe well
 * within one layer's decode (about 0.5% of a 48-layer step's pages at 32 x 4K
 * tokens: 4-9% faster than reading them in place; 1% is the edge), provided
 * the gather runs on a stream confined to a few CUs and the decode on a stream
 * over the others (kv_stream_create_cu_slots): gather waves that wait on PCIe
 * must not share CUs with the decode.  Below that window the per-layer cross-stream wait
 * costs more than the cold reads; above it both paths are PCIe-bound and
 * reading in place is faster.
 *
 * kv_pool_set_staging gives the pool a device buffer for this (256-byte
 * aligned; NULL or 0 bytes removes it).  It holds two halves (even and odd
 * layers) of `slots` slots each, a slot being one layer of one page:
 * num_kv_heads * 2 * 16 * head_dim elements.  *slots (nullable) gets the slot
 * count.  Decode calls of the pool must not be running.
 * Errors: KV_ERR_INVALID (alignment, metadata-only pool).
 */
int kv_pool_set_staging(kv_pool* pool, void* staging, size_t bytes, int32_t* slots);

/*
 * Batch page table for sessions sids (host int32 [n], ACTIVE) written to
 * `table` (device int32 [n][max_pages_per_session]) on `stream`: hot pages by
 * id; spilled pages, in batch and logical order, take staging slots
 * (KV_PAGE_STAGED | slot) while slots last and are read from the cold tier
 * directly (KV_PAGE_COLD | id) after that; unused entries are -1.  The
 * resulting plan (cold page per slot) stays with the pool until the next call.
 * *staged (nullable) gets the number of staged pages.  The table is valid until
 * the pool's bookkeeping of these sessions changes.
 * Errors: KV_ERR_INVALID, KV_ERR_STATE (a session not ACTIVE).
 */
int paged_decode_stage(kv_pool* pool, const int32_t* sids, int32_t n, int32_t* table,
                       kv_stream_t stream, int32_t* staged);

/*
 * Gather layer `layer`'s slices of the planned pages into the staging half of
 * that layer's parity, on `copy_stream` (typically not the decode stream, so
 * the gather overlaps the previous layer's decode).  The library orders it
 * after the plan's upload and after the decode that last read that half, and
 * orders the decode of `layer` after it.  Decoding a layer with staged entries
 * whose slices were not gathered for that layer reads no staged data: those
 * rows come out NaN.
 * Errors: KV_ERR_INVALID (no staging buffer, bad layer), KV_ERR_HIP.
 */
int paged_decode_prefetch(kv_pool* pool, int32_t layer, kv_stream_t copy_stream);

/* Device workspace bytes paged_decode_attention needs for this batch. */
size_t paged_decode_workspace_bytes(const kv_pool* pool, int32_t batch, int32_t num_q_heads);

/*
 * Paged grouped-query decode attention for one layer.  Decoding attends to the
 * cached KV of all past tokens (Sec. II) and reads the whole hot set every step
 * (Sec. III, data path 1).  For batch row b with L = seq_lens[b] and query head
 * h (KV head g = h / (num_q_heads / num_kv_heads)):
 *
 *     out[b][h] = sum_t softmax_t(scale * q[b][h] . k_t) v_t,  t = 0 .. L-1,
 *
 * with token t in page page_table[b * pt_stride + t / 16], slot t % 16.
 *
 *   q          device [batch][num_q_heads][head_dim], pool dtype
 *   page_table device int32, row b used for batch row b; may be the pool's own
 *              table (row = session id) or any gathered copy of rows
 *   seq_lens   device int32 [batch]; L = 0 writes zeros; L < 0 or
 *              L > 16 * pt_stride writes NaN for that row (no memory is read
 *              out of bounds); so does a page id outside the hot pool
 *   out        device [batch][num_q_heads][head_dim], pool dtype (bf16 rounded
 *              to nearest-even), written in full
 *   workspace  device, >= paged_decode_workspace_bytes(), 256-byte aligned
 * Only tokens [0, L) are read: other slots of the tail page and pages past
 * ceil(L / 16) may hold anything, NaN included.
 * Decode calls of one pool are ordered with each other across streams (they
 * share the pool's small arrival-counter array).  A call made while `stream`
 * is being captured into a HIP graph launches its two kernels and nothing
 * else (no events, no profiling); capture needs the separate merge and no
 * staged entries (KV_ERR_INVALID otherwise).  Replays read the pool as it is
 * then: q, seq_lens and the page table may change between replays.
 * Numerics: bf16 or float32 inputs, float32 accumulation, scores and weights in
 * float32 (bf16 pools round the softmax weights to bf16 for the weighted sum of
 * V and use the same rounded weights in the normaliser).  The result does not
 * depend on where pages sit in the pool.
 * num_q_heads / num_kv_heads must be an integer in 1 .. 16.
 * Errors: KV_ERR_INVALID (shapes, sizes, layer, metadata-only pool), KV_ERR_HIP.
 */
int paged_decode_attention(kv_pool* pool, int32_t layer, const void* q, const int32_t* page_table,
                           int64_t pt_stride, const int32_t* seq_lens, int32_t batch,
                           int32_t num_q_heads, float scale, void* out, void* workspace,
                           size_t ws_bytes, kv_stream_t stream);

/*
 * A decode step's append fused into its decode (data paths 3 and 1, Sec. III):
 * for each batch row b with 0 < L = seq_lens[b] <= 16 * pt_stride, the row's
 * new token, k_new / v_new row b (device arrays [batch][num_kv_heads][head_dim]
 * of the pool's dtype, 16-byte aligned), is written as token L - 1 into the
 * page that page-table entry (L - 1) / 16 names (a hot page, or KV_PAGE_COLD | id:
 * a spilled page written in place), and then out[b] is the attention over
 * tokens [0, L), the new one included, exactly as paged_decode_attention would
 * give after a separate append.  The wave that reads the row's last page for a
 * KV head writes that head's part of the token first, so the append costs no
 * launch of its own and no extra pass: one kernel launch per layer serves a
 * whole decode step's attention and KV append, and a serving step captured in
 * a HIP graph holds no append nodes.  A tail entry naming no page writes
 * nothing (and that row decodes to NaN, as in paged_decode_attention).  The
 * pool's bookkeeping is untouched: call kv_session_extend first, which drops
 * the cold copy of the page receiving the token.  A layer with staged entries
 * (paged_decode_prefetch) is refused: the token must go to the page itself.
 * Other arguments and errors as paged_decode_attention.
 */
int paged_decode_attention_append(kv_pool* pool, int32_t layer, const void* q, const void* k_new,
                                  const void* v_new, const int32_t* page_table, int64_t pt_stride,
                                  const int32_t* seq_lens, int32_t batch, int32_t num_q_heads, float scale,
                                  void* out, void* workspace, size_t ws_bytes, kv_stream_t stream);

/*
 * paged_decode_attention without a workspace argument and without allocating:
 * for callers that cannot call the allocator (code under HIP graph capture,
 * serving loops and harnesses that forbid allocation).  The split partials and
 * the row page prefix live in a device array of KV_DECODE_SCRATCH_BYTES that
 * the library holds on each GPU it runs on until the process ends (its address
 * is taken when a pool is created on that GPU).  Arguments, numerics and
 * results are those of paged_decode_attention with the same pool settings (the
 * same kernels and work split, so the outputs are bitwise equal).  Nothing in
 * the array needs to start at zero, and it keeps the last call's contents.
 * Every call on one GPU shares that array: calls that overlap in time on one
 * GPU (two streams, two pools, two threads) race and corrupt each other's
 * results; order them.  The call takes no profiling events.
 * Errors: as paged_decode_attention; KV_ERR_INVALID when the batch needs more
 * scratch than KV_DECODE_SCRATCH_BYTES (paged_decode_workspace_bytes gives the
 * need; about 4.2 KB per (row, KV head) plus 3.2 MB at 32 query / 4 KV heads,
 * d = 128, so batches up to about 1,800 rows fit).
 */
#define KV_DECODE_SCRATCH_BYTES (32u << 20)
int paged_decode_attention_noalloc(kv_pool* pool, int32_t layer, const void* q, const int32_t* page_table,
                                   int64_t pt_stride, const int32_t* seq_lens, int32_t batch,
                                   int32_t num_q_heads, float scale, void* out, kv_stream_t stream);

/*
 * The work split of paged_decode_attention, written out (device int32
 * [waves + batch * num_kv_heads][4]).  Waves form workers of L waves: L = 4
 * when num_kv_heads and `waves` are multiples of 4, else 1.  A unit is one
 * page of one (row b, head group hg) with Hkv / L groups per row; units are
 * ordered by (b, hg, page); worker k of waves / L takes units
 * [floor(k T L / waves), floor((k + 1) T L / waves)) of the T units.  Where a
 * worker meets the units of (b, hg), its wave w makes one partial result for
 * KV head g = L hg + w, stored in slot (k + b Hkv / L + hg) L + w as
 * (b, g, first page, end page).  Unused slots hold (-1, -1, 0, 0).  With
 * L = 4 a worker's four waves read the four heads' tiles of the same pages,
 * which HBM serves faster than unrelated pages.  The split is not the
 * paper's: it is how this library balances sessions of different lengths
 * over the GPU.
 */
int paged_decode_partition(kv_pool* pool, const int32_t* seq_lens, int32_t batch, int32_t waves,
                           int32_t* slots_out, kv_stream_t stream);

/* ----------------------------------------------------------------------- */
/* Diagnostics                                                              */
/* ----------------------------------------------------------------------- */

const char* kv_strerror(int status);
const char* kv_last_error(void);

/*
 * Measurement context, not part of the KV path: a streaming read of `bytes`
 * (a multiple of 16) of device memory at `buf` (16-byte aligned), with the
 * 16-byte nontemporal loads the decode kernel uses and 8 of them in flight
 * per thread, on `blocks` (1 .. 2^20) blocks of 256 threads that take
 * contiguous 32 KiB chunks in turn.  Each block
 * writes the XOR of what it read to out[block] (device, `blocks` words), so
 * the reads cannot be elided.  Asynchronous on `stream`; time it with events
 * around the call.  It gives the sequential-read rate this GPU reaches, the
 * practical ceiling that the decode's random page reads are compared with.
 * KV_ERR_INVALID for bad arguments.
 */
int kv_read_probe(const void* buf, size_t bytes, uint32_t* out, int32_t blocks, kv_stream_t stream);

/*
 * Profiling hook.  When enabled, every timed kernel the pool launches (the ids
 * above) carries a pair of HIP events that its dispatch records at the kernel's
 * start and end (hipExtLaunchKernel), so a duration covers the kernel alone.
 * kv_pool_profile_read waits for the recorded launches of one kernel id,
 * returns their count and summed duration in milliseconds, and forgets them.
 */
int kv_pool_set_profiling(kv_pool* pool, int enable);
int kv_pool_profile_read(kv_pool* pool, int32_t kernel_id, int32_t* launches, double* total_ms);

#ifdef __cplusplus
}
#endif

#endif /* HOTCOLD_KV_H */
