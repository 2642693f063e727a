// Host runtime of the hot-cold KV library: pool bookkeeping, session state
// machine, deterministic page allocation and the C ABI declared in hotcold_kv.h.
//
// Bookkeeping lives on the host.  Device work (page copies, page-table writes,
// decode) is enqueued on the caller's stream through the launchers in
// kernels.h.  Every call validates and plans first and commits its bookkeeping
// only after its device work was enqueued, so a failing call changes nothing.

#include "hotcold_kv.h"
#include "kernels.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <new>
#include <string>
#include <vector>

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

int hip_fail(hipError_t e, const char* what) {
    return fail(KV_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Free-page set with lowest-id-first allocation (a bitmap; bit set = free).
class PageSet {
  public:
    void init(int32_t n) {
        n_ = n;
        free_ = n;
        bits_.assign((static_cast<size_t>(n) + 63) / 64, ~0ull);
        if (n % 64) bits_.back() = (1ull << (n % 64)) - 1;
        hint_ = 0;
    }
    int32_t size() const { return n_; }
    int32_t free_count() const { return free_; }
    bool is_free(int32_t p) const { return (bits_[p >> 6] >> (p & 63)) & 1ull; }
    void take(int32_t p) {
        bits_[p >> 6] &= ~(1ull << (p & 63));
        --free_;
    }
    void give(int32_t p) {
        bits_[p >> 6] |= 1ull << (p & 63);
        ++free_;
        if (static_cast<size_t>(p >> 6) < hint_) hint_ = p >> 6;
    }
    // The k lowest free ids, ascending, without taking them.
    void lowest(int32_t k, std::vector<int32_t>& out) {
        out.clear();
        out.reserve(k);
        while (hint_ < bits_.size() && bits_[hint_] == 0) ++hint_;
        for (size_t w = hint_; w < bits_.size() && static_cast<int32_t>(out.size()) < k; ++w) {
            uint64_t x = bits_[w];
            while (x && static_cast<int32_t>(out.size()) < k) {
                const int b = __builtin_ctzll(x);
                out.push_back(static_cast<int32_t>(w * 64 + b));
                x &= x - 1;
            }
        }
    }

  private:
    std::vector<uint64_t> bits_;
    int32_t n_ = 0, free_ = 0;
    size_t hint_ = 0;
};

struct Session {
    int32_t state = KV_SESSION_FREE;
    int32_t seq_len = 0;
    int64_t stamp = 0;          // pause time (LRU order) while PAUSED
    std::vector<int32_t> hot;   // hot page per logical page, -1 = not resident
    std::vector<int32_t> cold;  // cold page per logical page, -1 = no valid copy
    std::vector<uint8_t> spilled;  // 1: the row entry names the cold page (spill)
};

// One resident page of a paused session chosen for eviction.
struct Victim {
    int32_t sid, page;
};

// Hot pages for one call, and what must be evicted to free them.
struct Alloc {
    std::vector<Victim> victims;       // LRU pages evicted first
    std::vector<int32_t> victim_cold;  // cold page for each victim without a valid copy
    std::vector<int32_t> pages;        // hot pages handed out, ascending
    std::vector<int32_t> spill_cold;   // fresh cold pages for the pages that spill
};

constexpr int kStagingSlots = 4;
constexpr size_t kStagingBytes = size_t(1) << 20;
constexpr int32_t kStagingEntries = static_cast<int32_t>(kStagingBytes / sizeof(hck::CopyEntry));
constexpr int32_t kMaxDecodeBatch = hck::kMaxDecodeBatch;
#ifndef HCK_DECODE_WAVES_PER_CU
#define HCK_DECODE_WAVES_PER_CU 3
#endif
constexpr int32_t kDecodeWavesPerCu = HCK_DECODE_WAVES_PER_CU;

struct StagingSlot {
    void* host = nullptr;  // pinned
    void* dev = nullptr;
    hipEvent_t done = nullptr;
    bool pending = false;
};

struct ProfRec {
    hipEvent_t start, stop;
};

int32_t pages_of(int64_t seq_len) {
    return static_cast<int32_t>((seq_len + KV_PAGE_TOKENS - 1) / KV_PAGE_TOKENS);
}

size_t elt_size(int32_t dtype) { return dtype == KV_DTYPE_BF16 ? 2 : 4; }

size_t layout_page_bytes(const kv_pool_desc* d) {
    return static_cast<size_t>(d->num_layers) * d->num_kv_heads * 2 * KV_PAGE_TOKENS * d->head_dim *
           elt_size(d->dtype);
}

bool desc_valid(const kv_pool_desc* d) {
    return d && d->num_layers >= 1 && d->num_layers <= 64 && d->num_kv_heads >= 1 &&
           d->num_kv_heads <= 16 && (d->head_dim == 64 || d->head_dim == 128) &&
           d->page_size == KV_PAGE_TOKENS &&
           (d->dtype == KV_DTYPE_BF16 || d->dtype == KV_DTYPE_F32) && d->num_hot_pages >= 0 &&
           d->num_cold_pages >= 0 &&
           (d->cold_location == KV_COLD_DEVICE || d->cold_location == KV_COLD_PINNED_HOST) &&
           d->max_sessions >= 1 && d->max_pages_per_session >= 1 &&
           static_cast<int64_t>(d->max_sessions) * d->max_pages_per_session < (int64_t(1) << 31) &&
           d->max_pages_per_session <= kStagingEntries;
}

class DeviceGuard {
  public:
    explicit DeviceGuard(int dev) {
        if (hipGetDevice(&prev_) == hipSuccess && prev_ != dev) {
            changed_ = hipSetDevice(dev) == hipSuccess;
        }
    }
    ~DeviceGuard() {
        if (changed_) (void)hipSetDevice(prev_);
    }

  private:
    int prev_ = -1;
    bool changed_ = false;
};

}  // namespace

struct kv_pool {
    kv_pool_desc d{};
    bool meta = false;
    char* hot = nullptr;
    char* cold = nullptr;  // device-visible address of the cold pool
    int32_t* pt = nullptr;
    int64_t page_bytes = 0;
    PageSet hot_free, cold_free;
    std::vector<int32_t> cold_ref;
    std::vector<Session> sessions;
    int64_t clock = 0;                // pause stamps
    std::map<int64_t, int32_t> lru;  // stamp -> sid of paused sessions with resident pages
    kv_pool_stats_t st{};
    int cus = 0;
    int32_t waves_override = 0;
    int32_t copy_blocks = 0;  // cap of the page-copy grid (0: default)
    bool spill = false;       // place pages in the cold tier instead of failing
    // staging of spilled pages for decode (one layer's slices, two halves)
    char* stage = nullptr;
    int32_t stage_slots = 0;  // slots per half
    int64_t slice_bytes = 0;  // one layer of one page
    std::vector<int32_t> plan;            // cold page per staging slot
    hck::CopyEntry* plan_dev = nullptr;   // the plan as copy entries (device)
    hck::CopyEntry* plan_host = nullptr;  // pinned upload buffer of the plan
    int32_t plan_cap = 0;
    hipEvent_t plan_ready = nullptr, prefetch_done = nullptr;
    bool plan_ready_pending = false, prefetch_pending = false;
    hipEvent_t half_ready[2] = {nullptr, nullptr}, half_free[2] = {nullptr, nullptr};
    bool half_ready_pending[2] = {false, false}, half_free_pending[2] = {false, false};
    int32_t half_layer[2] = {-1, -1};     // layer gathered into each half for the current plan
    StagingSlot ring[kStagingSlots];
    int ring_next = 0;
    // One event per stream on which calls freed hot pages: recorded after the
    // last such call's device work on that stream.
    struct FreeMark {
        hipStream_t stream;
        hipEvent_t event;
    };
    std::vector<FreeMark> free_marks;
    bool profiling = false;
    int32_t combine_mode = KV_COMBINE_SEPARATE;
    char* cold_host = nullptr;      // host address of a pinned-host cold pool (null otherwise)
    // Pool geometries: the hot pool is layer-major (one layer's slices of all
    // pages together: a decode reads within 1 / num_layers of it), the cold
    // pool page-major (each 16-token block contiguous).
    hck::PoolGeom hot_geom, cold_geom;
    int32_t host_copy = KV_HOST_COPY_DMA;
    int32_t compute_mode = KV_DECODE_MATRIX;
    int32_t* counters = nullptr;  // decode arrival counters, zero between calls
    void* scratch = nullptr;      // the no-allocation decode's device array on this pool's device
    hipEvent_t decode_event = nullptr;
    bool decode_pending = false;
    std::vector<ProfRec> prof[KV_KERNEL_COUNT];
    std::vector<hipEvent_t> spare_events;

    ~kv_pool() {
        if (meta) return;
        DeviceGuard g(d.device);
        for (auto& s : ring) {
            if (s.done) (void)hipEventSynchronize(s.done);
            if (s.host) (void)hipHostFree(s.host);
            if (s.dev) (void)hipFree(s.dev);
            if (s.done) (void)hipEventDestroy(s.done);
        }
        for (const FreeMark& m : free_marks) (void)hipEventDestroy(m.event);
        if (decode_event) {
            (void)hipEventSynchronize(decode_event);
            (void)hipEventDestroy(decode_event);
        }
        if (counters) (void)hipFree(counters);
        for (auto& v : prof)
            for (auto& r : v) {
                (void)hipEventDestroy(r.start);
                (void)hipEventDestroy(r.stop);
            }
        for (auto e : spare_events) (void)hipEventDestroy(e);
        free_staging_state();
        for (hipEvent_t e : {plan_ready, prefetch_done, half_ready[0], half_ready[1], half_free[0],
                             half_free[1]})
            if (e) (void)hipEventDestroy(e);
    }

    // Wait for every use of the plan buffers, then free them.
    void free_staging_state() {
        if (prefetch_pending) (void)hipEventSynchronize(prefetch_done);
        if (plan_ready_pending) (void)hipEventSynchronize(plan_ready);
        for (int b = 0; b < 2; ++b)
            if (half_free_pending[b]) (void)hipEventSynchronize(half_free[b]);
        prefetch_pending = plan_ready_pending = false;
        half_free_pending[0] = half_free_pending[1] = false;
        half_ready_pending[0] = half_ready_pending[1] = false;
        if (plan_dev) (void)hipFree(plan_dev);
        if (plan_host) (void)hipHostFree(plan_host);
        plan_dev = nullptr;
        plan_host = nullptr;
        plan_cap = 0;
        plan.clear();
        half_layer[0] = half_layer[1] = -1;
    }

    bool tiered() const { return spill || stage_slots > 0; }

    hipStream_t strm(kv_stream_t s) const { return static_cast<hipStream_t>(s); }

    // Make `stream` wait for the device work of every call that freed hot pages,
    // on whichever stream it ran.
    int order_after_frees(hipStream_t s) {
        for (const FreeMark& m : free_marks) {
            hipError_t e = hipStreamWaitEvent(s, m.event, 0);
            if (e != hipSuccess) return hip_fail(e, "hipStreamWaitEvent");
        }
        return KV_OK;
    }

    // After a call that freed hot pages enqueued its work on `s`.  Marks of other
    // streams whose work has finished are dropped; a single shared event would
    // lose the work of the previous freeing call whenever streams alternate.
    int note_frees(hipStream_t s) {
        size_t keep = 0;
        for (size_t i = 0; i < free_marks.size(); ++i) {
            const FreeMark m = free_marks[i];
            if (m.stream != s && hipEventQuery(m.event) == hipSuccess) {
                (void)hipEventDestroy(m.event);
                continue;
            }
            free_marks[keep++] = m;
        }
        free_marks.resize(keep);
        FreeMark* mine = nullptr;
        for (FreeMark& m : free_marks)
            if (m.stream == s) mine = &m;
        if (!mine) {
            hipEvent_t ev = nullptr;
            hipError_t e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
            if (e != hipSuccess) return hip_fail(e, "hipEventCreateWithFlags");
            free_marks.push_back(FreeMark{s, ev});
            mine = &free_marks.back();
        }
        hipError_t e = hipEventRecord(mine->event, s);
        if (e != hipSuccess) return hip_fail(e, "hipEventRecord");
        return KV_OK;
    }

    int acquire_slot(StagingSlot** out) {
        StagingSlot& s = ring[ring_next];
        ring_next = (ring_next + 1) % kStagingSlots;
        if (s.pending) {
            hipError_t e = hipEventSynchronize(s.done);
            if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize(staging)");
            s.pending = false;
        }
        *out = &s;
        return KV_OK;
    }

    hipEvent_t take_event() {
        if (!spare_events.empty()) {
            hipEvent_t e = spare_events.back();
            spare_events.pop_back();
            return e;
        }
        hipEvent_t e = nullptr;
        if (hipEventCreate(&e) != hipSuccess) return nullptr;
        return e;
    }

    // Events for one launch when profiling is on: the launch records them at
    // its kernel's start and end.  prof_done files them under `kernel` if the
    // launch went out, or returns them to the spares.
    hck::LaunchEvents prof_events() {
        hck::LaunchEvents ev;
        if (!profiling) return ev;
        ev.start = take_event();
        ev.stop = take_event();
        if (!ev.start || !ev.stop) {
            if (ev.start) spare_events.push_back(ev.start);
            if (ev.stop) spare_events.push_back(ev.stop);
            return hck::LaunchEvents{};
        }
        return ev;
    }
    void prof_done(int kernel, const hck::LaunchEvents& ev, hipError_t launched) {
        if (!ev.start) return;
        if (launched == hipSuccess) {
            prof[kernel].push_back(ProfRec{ev.start, ev.stop});
        } else {
            spare_events.push_back(ev.start);
            spare_events.push_back(ev.stop);
        }
    }

    // Enqueue whole-page copies between the pools (in chunks that fit a
    // staging slot): cold -> hot when to_hot, else hot -> cold.  Entries that
    // only write the page table (rows cleared on eviction, resident pages
    // remapped on resume) go to the table-write kernel instead, so the copy
    // grid only walks pages that move.
    int submit_copies(bool to_hot, const std::vector<hck::CopyEntry>& all, hipStream_t s, int kernel_id) {
        std::vector<hck::CopyEntry> entries, writes;
        entries.reserve(all.size());
        for (const hck::CopyEntry& e : all) {
            if (e.src >= 0)
                entries.push_back(e);
            else if (e.pt_index >= 0)
                writes.push_back(e);
        }
        if (!writes.empty()) {
            int rc = submit_table_writes(writes, s);
            if (rc) return rc;
        }
        if (cold_host && host_copy == KV_HOST_COPY_DMA) return submit_dma_copies(to_hot, entries, s, kernel_id);
        const hck::PoolGeom& src = to_hot ? cold_geom : hot_geom;
        const hck::PoolGeom& dst = to_hot ? hot_geom : cold_geom;
        for (size_t off = 0; off < entries.size(); off += kStagingEntries) {
            const int32_t n = static_cast<int32_t>(
                std::min<size_t>(kStagingEntries, entries.size() - off));
            StagingSlot* slot;
            int rc = acquire_slot(&slot);
            if (rc) return rc;
            std::memcpy(slot->host, entries.data() + off, n * sizeof(hck::CopyEntry));
            hipError_t e = hipMemcpyAsync(slot->dev, slot->host, n * sizeof(hck::CopyEntry),
                                          hipMemcpyHostToDevice, s);
            if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync(copy list)");
            const hck::LaunchEvents ev = prof_events();
            e = hck::launch_page_copy(src, dst, slice_bytes, d.num_layers, /*by_layer=*/!to_hot,
                                      static_cast<const hck::CopyEntry*>(slot->dev), n, pt, copy_blocks, s, ev);
            prof_done(kernel_id, ev, e);
            if (e != hipSuccess) return hip_fail(e, "page copy launch");
            e = hipEventRecord(slot->done, s);
            if (e != hipSuccess) return hip_fail(e, "hipEventRecord(staging)");
            slot->pending = true;
        }
        return KV_OK;
    }

    // Page copies to or from a pinned-host cold pool on the DMA engines, then
    // the page-table entries (stream-ordered after the copies).  A copy kernel
    // reading or writing host memory keeps its waves waiting on PCIe in the
    // CUs' memory pipelines, which slows a decode running on another stream
    // many times over; the DMA engines use no CU.  A host page is contiguous
    // and a hot page is one slice per layer.  A run of k pages consecutive on
    // both sides is min(k, num_layers) 2D copies: one per page (num_layers
    // rows of one slice), or for long runs one per layer (k rows of one slice,
    // contiguous in the hot pool, a page apart in host memory).
    int submit_dma_copies(bool to_hot, const std::vector<hck::CopyEntry>& entries, hipStream_t s, int kernel_id) {
        if (entries.empty()) return KV_OK;
        const hipMemcpyKind kind = to_hot ? hipMemcpyHostToDevice : hipMemcpyDeviceToHost;
        const size_t slice = static_cast<size_t>(slice_bytes);
        const hck::LaunchEvents ev = prof_events();
        hipError_t e = ev.start ? hipEventRecord(ev.start, s) : hipSuccess;
        auto copy2d = [&](char* hot_p, size_t hot_pitch, char* host_p, size_t host_pitch, size_t rows) {
            return to_hot ? hipMemcpy2DAsync(hot_p, hot_pitch, host_p, host_pitch, slice, rows, kind, s)
                          : hipMemcpy2DAsync(host_p, host_pitch, hot_p, hot_pitch, slice, rows, kind, s);
        };
        for (size_t i = 0; i < entries.size() && e == hipSuccess;) {
            size_t j = i + 1;
            while (j < entries.size() && entries[j].src == entries[j - 1].src + 1 &&
                   entries[j].dst == entries[j - 1].dst + 1)
                ++j;
            const size_t k = j - i;
            const int32_t hp = to_hot ? entries[i].dst : entries[i].src;
            const int32_t cp = to_hot ? entries[i].src : entries[i].dst;
            char* host_p = cold_host + static_cast<int64_t>(cp) * page_bytes;
            if (k >= static_cast<size_t>(d.num_layers)) {
                for (int32_t l = 0; l < d.num_layers && e == hipSuccess; ++l)
                    e = copy2d(hck::slice_at(hot_geom, hp, l), slice, host_p + l * slice, page_bytes, k);
            } else {
                for (size_t m = 0; m < k && e == hipSuccess; ++m)
                    e = copy2d(hck::slice_at(hot_geom, hp + static_cast<int32_t>(m), 0), hot_geom.layer_stride,
                               host_p + m * page_bytes, slice, d.num_layers);
            }
            i = j;
        }
        if (e == hipSuccess && ev.stop) e = hipEventRecord(ev.stop, s);
        prof_done(kernel_id, ev, e);
        if (e != hipSuccess) return hip_fail(e, "hipMemcpy2DAsync(host-tier pages)");
        std::vector<hck::CopyEntry> writes;
        for (const hck::CopyEntry& c : entries)
            if (c.pt_index >= 0) writes.push_back(hck::CopyEntry{-1, -1, c.pt_index, c.pt_value});
        return writes.empty() ? KV_OK : submit_table_writes(writes, s);
    }

    int submit_table_writes(const std::vector<hck::CopyEntry>& entries, hipStream_t s) {
        for (size_t off = 0; off < entries.size(); off += kStagingEntries) {
            const int32_t n = static_cast<int32_t>(std::min<size_t>(kStagingEntries, entries.size() - off));
            StagingSlot* slot;
            int rc = acquire_slot(&slot);
            if (rc) return rc;
            std::memcpy(slot->host, entries.data() + off, n * sizeof(hck::CopyEntry));
            hipError_t e = hipMemcpyAsync(slot->dev, slot->host, n * sizeof(hck::CopyEntry),
                                          hipMemcpyHostToDevice, s);
            if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync(table writes)");
            e = hck::launch_table_writes(static_cast<const hck::CopyEntry*>(slot->dev), n, pt, s);
            if (e != hipSuccess) return hip_fail(e, "table write launch");
            e = hipEventRecord(slot->done, s);
            if (e != hipSuccess) return hip_fail(e, "hipEventRecord(staging)");
            slot->pending = true;
        }
        return KV_OK;
    }

    // Write `n` page ids into page-table row `sid` (entries 0..n-1).
    int submit_row(int32_t sid, const int32_t* vals, int32_t n, hipStream_t s) {
        if (n <= 0) return KV_OK;
        StagingSlot* slot;
        int rc = acquire_slot(&slot);
        if (rc) return rc;
        std::memcpy(slot->host, vals, n * sizeof(int32_t));
        hipError_t e = hipMemcpyAsync(pt + static_cast<int64_t>(sid) * d.max_pages_per_session,
                                      slot->host, n * sizeof(int32_t), hipMemcpyHostToDevice, s);
        if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync(page-table row)");
        e = hipEventRecord(slot->done, s);
        if (e != hipSuccess) return hip_fail(e, "hipEventRecord(staging)");
        slot->pending = true;
        return KV_OK;
    }

    int clear_row(int32_t sid, int32_t n, hipStream_t s) {
        if (n <= 0) return KV_OK;
        hipError_t e =
            hck::launch_fill_i32(pt + static_cast<int64_t>(sid) * d.max_pages_per_session, n, -1, s);
        if (e != hipSuccess) return hip_fail(e, "page-table clear");
        return KV_OK;
    }

    // Write `n` page ids into page-table row `sid` starting at entry `first`.
    int submit_row_at(int32_t sid, int32_t first, const int32_t* vals, int32_t n, hipStream_t s) {
        if (n <= 0) return KV_OK;
        StagingSlot* slot;
        int rc = acquire_slot(&slot);
        if (rc) return rc;
        std::memcpy(slot->host, vals, n * sizeof(int32_t));
        hipError_t e = hipMemcpyAsync(
            pt + static_cast<int64_t>(sid) * d.max_pages_per_session + first, slot->host,
            n * sizeof(int32_t), hipMemcpyHostToDevice, s);
        if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync(page-table row)");
        e = hipEventRecord(slot->done, s);
        if (e != hipSuccess) return hip_fail(e, "hipEventRecord(staging)");
        slot->pending = true;
        return KV_OK;
    }

    static bool has_resident(const Session& s) {
        for (int32_t p : s.hot)
            if (p >= 0) return true;
        return false;
    }

    static bool has_row_entries(const Session& s) {
        for (size_t i = 0; i < s.hot.size(); ++i)
            if (s.hot[i] >= 0 || s.spilled[i]) return true;
        return false;
    }

    // Page-table entries of new pages: hot ids, then the spilled pages' cold ids.
    static std::vector<int32_t> new_entries(const Alloc& a) {
        std::vector<int32_t> v(a.pages);
        for (int32_t c : a.spill_cold) v.push_back(c | KV_PAGE_COLD);
        return v;
    }

    // Least-recently-used resident pages of paused sessions: oldest pause first,
    // lowest logical page first, skipping `exclude`; at most `need` of them.
    void plan_lru(int64_t need, const std::vector<int32_t>& exclude, std::vector<Victim>& out) const {
        out.clear();
        for (auto it = lru.begin(); it != lru.end() && static_cast<int64_t>(out.size()) < need; ++it) {
            const int32_t sid = it->second;
            if (std::find(exclude.begin(), exclude.end(), sid) != exclude.end()) continue;
            const Session& s = sessions[sid];
            for (size_t i = 0; i < s.hot.size() && static_cast<int64_t>(out.size()) < need; ++i)
                if (s.hot[i] >= 0) out.push_back(Victim{sid, static_cast<int32_t>(i)});
        }
    }

    // Cold pages for the victims that have no valid cold copy (write-on-evict).
    int plan_victim_cold(Alloc& a) {
        int64_t dirty = 0;
        for (const Victim& v : a.victims) dirty += sessions[v.sid].cold[v.page] < 0;
        if (dirty > cold_free.free_count())
            return fail(KV_ERR_NO_COLD_PAGES, "evicting %zu pages needs %lld cold pages, %d free",
                        a.victims.size(), static_cast<long long>(dirty), cold_free.free_count());
        cold_free.lowest(static_cast<int32_t>(dirty), a.victim_cold);
        return KV_OK;
    }

    // Plan k pages, evicting LRU pages of paused sessions (never those of
    // `exclude`) when too few hot pages are free.  Without spill all k are hot
    // or the call fails; with spill (the pool's, or `allow_spill`) the pages
    // that find no hot page spill: fresh cold pages if `fresh_spill`, else they
    // stay where they are.  Changes nothing.
    int plan_alloc(int64_t k, const std::vector<int32_t>& exclude, Alloc& a, bool fresh_spill = true,
                   bool allow_spill = false) {
        a = Alloc();
        const int64_t have = hot_free.free_count();
        if (k <= have) {
            hot_free.lowest(static_cast<int32_t>(k), a.pages);
            return KV_OK;
        }
        plan_lru(k - have, exclude, a.victims);
        const int64_t short_by = k - have - static_cast<int64_t>(a.victims.size());
        if (short_by > 0 && !(spill || allow_spill))
            return fail(KV_ERR_NO_HOT_PAGES, "need %lld hot pages: %lld free, %zu evictable",
                        static_cast<long long>(k), static_cast<long long>(have), a.victims.size());
        const int64_t n_hot = k - std::max<int64_t>(short_by, 0);
        const int64_t n_spill = fresh_spill ? std::max<int64_t>(short_by, 0) : 0;
        int64_t dirty = 0;
        for (const Victim& v : a.victims) dirty += sessions[v.sid].cold[v.page] < 0;
        if (dirty + n_spill > cold_free.free_count())
            return fail(KV_ERR_NO_COLD_PAGES, "need %lld cold pages (%lld evicted, %lld spilled), %d free",
                        static_cast<long long>(dirty + n_spill), static_cast<long long>(dirty),
                        static_cast<long long>(n_spill), cold_free.free_count());
        std::vector<int32_t> both;
        cold_free.lowest(static_cast<int32_t>(dirty + n_spill), both);
        a.victim_cold.assign(both.begin(), both.begin() + dirty);
        a.spill_cold.assign(both.begin() + dirty, both.end());
        PageSet after = hot_free;
        for (const Victim& v : a.victims) after.give(sessions[v.sid].hot[v.page]);
        after.lowest(static_cast<int32_t>(n_hot), a.pages);
        return KV_OK;
    }

    void commit_spill(const Alloc& a) {
        for (int32_t c : a.spill_cold) {
            cold_free.take(c);
            cold_ref[c] = 1;
        }
        st.spilled_pages += static_cast<int64_t>(a.spill_cold.size());
    }

    // Enqueue the victims' cold writes and row clears (one launch), before any
    // launch that reuses their hot pages on the same stream.
    int submit_victims(const Alloc& a, hipStream_t s) {
        if (a.victims.empty()) return KV_OK;
        std::vector<hck::CopyEntry> entries;
        entries.reserve(a.victims.size());
        size_t k = 0;
        for (const Victim& v : a.victims) {
            const Session& ss = sessions[v.sid];
            const bool copy = ss.cold[v.page] < 0;
            entries.push_back(hck::CopyEntry{copy ? ss.hot[v.page] : -1, copy ? a.victim_cold[k] : -1,
                                             v.sid * d.max_pages_per_session + v.page, -1});
            k += copy;
        }
        int rc = submit_copies(false, entries, s, KV_KERNEL_EVICT_COPY);
        if (!rc) rc = note_frees(s);
        return rc;
    }

    void commit_victims(const Alloc& a) {
        size_t k = 0;
        for (const Victim& v : a.victims) {
            Session& ss = sessions[v.sid];
            if (ss.cold[v.page] < 0) {
                const int32_t c = a.victim_cold[k++];
                cold_free.take(c);
                cold_ref[c] = 1;
                ss.cold[v.page] = c;
                st.pages_to_cold += 1;
                st.bytes_to_cold += page_bytes;
            }
            hot_free.give(ss.hot[v.page]);
            ss.hot[v.page] = -1;
            st.lru_evicted_pages += 1;
        }
        for (const Victim& v : a.victims) {
            Session& ss = sessions[v.sid];
            if (!has_resident(ss)) lru.erase(ss.stamp);
        }
    }

    int32_t new_sid() const {
        for (int32_t i = 0; i < d.max_sessions; ++i)
            if (sessions[i].state == KV_SESSION_FREE) return i;
        return -1;
    }

    Session* session(int32_t sid) {
        if (sid < 0 || sid >= d.max_sessions) return nullptr;
        return &sessions[sid];
    }

    void release_cold(int32_t c) {
        if (--cold_ref[c] == 0) cold_free.give(c);
    }

    // Three waves per CU: enough loads in flight to saturate HBM with the
    // register ring, without the extra partials and DRAM contention of more.
    int32_t auto_waves() const { return std::max<int32_t>(cus * kDecodeWavesPerCu, 1); }
    int32_t decode_waves() const { return waves_override > 0 ? waves_override : auto_waves(); }
};

extern "C" {

size_t kv_page_bytes(const kv_pool_desc* desc) {
    if (!desc_valid(desc)) return 0;
    return layout_page_bytes(desc);
}

int kv_pool_create(const kv_pool_desc* desc, void* hot_base, size_t hot_bytes, void* cold_base,
                   size_t cold_bytes, int32_t* page_table, kv_stream_t stream, kv_pool** out) {
    if (!out) return fail(KV_ERR_INVALID, "out is NULL");
    *out = nullptr;
    if (!desc_valid(desc)) return fail(KV_ERR_INVALID, "invalid pool descriptor");
    const bool meta = (desc->flags & KV_POOL_METADATA_ONLY) != 0;
    const size_t pb = layout_page_bytes(desc);
    if (!meta) {
        if (desc->num_hot_pages > 0 && (!hot_base || hot_bytes < pb * desc->num_hot_pages))
            return fail(KV_ERR_INVALID, "hot pool smaller than %d pages of %zu bytes",
                        desc->num_hot_pages, pb);
        if (desc->num_cold_pages > 0 && (!cold_base || cold_bytes < pb * desc->num_cold_pages))
            return fail(KV_ERR_INVALID, "cold pool smaller than %d pages of %zu bytes",
                        desc->num_cold_pages, pb);
        if (!page_table) return fail(KV_ERR_INVALID, "page table is NULL");
        if ((reinterpret_cast<uintptr_t>(hot_base) | reinterpret_cast<uintptr_t>(cold_base)) & 255)
            return fail(KV_ERR_INVALID, "pools must be 256-byte aligned");
    }
    kv_pool* p = new (std::nothrow) kv_pool();
    if (!p) return fail(KV_ERR_OOM, "out of host memory");
    p->d = *desc;
    p->meta = meta;
    p->page_bytes = static_cast<int64_t>(pb);
    p->slice_bytes = static_cast<int64_t>(pb) / desc->num_layers;
    p->hot_free.init(desc->num_hot_pages);
    p->cold_free.init(desc->num_cold_pages);
    p->cold_ref.assign(desc->num_cold_pages, 0);
    p->sessions.assign(desc->max_sessions, Session());
    if (!meta) {
        DeviceGuard g(desc->device);
        p->hot = static_cast<char*>(hot_base);
        p->pt = page_table;
        hipError_t e = hipSuccess;
        if (desc->cold_location == KV_COLD_PINNED_HOST && cold_base) {
            void* dp = nullptr;
            e = hipHostGetDevicePointer(&dp, cold_base, 0);
            if (e != hipSuccess) {
                delete p;
                return hip_fail(e, "hipHostGetDevicePointer(cold pool)");
            }
            p->cold = static_cast<char*>(dp);
            p->cold_host = static_cast<char*>(cold_base);
        } else {
            p->cold = static_cast<char*>(cold_base);
        }
        p->hot_geom = hck::PoolGeom{p->hot, p->slice_bytes, p->slice_bytes * desc->num_hot_pages};
        p->cold_geom = hck::PoolGeom{p->cold, p->page_bytes, p->slice_bytes};
        e = hipDeviceGetAttribute(&p->cus, hipDeviceAttributeMultiprocessorCount, desc->device);
        if (e != hipSuccess) {
            delete p;
            return hip_fail(e, "hipDeviceGetAttribute");
        }
        for (auto& s : p->ring) {
            if (hipHostMalloc(&s.host, kStagingBytes, hipHostMallocDefault) != hipSuccess ||
                hipMalloc(&s.dev, kStagingBytes) != hipSuccess ||
                hipEventCreateWithFlags(&s.done, hipEventDisableTiming) != hipSuccess) {
                delete p;
                return fail(KV_ERR_OOM, "staging allocation failed");
            }
        }
        if (hipEventCreateWithFlags(&p->decode_event, hipEventDisableTiming) != hipSuccess) {
            delete p;
            return fail(KV_ERR_OOM, "event creation failed");
        }
        e = hck::scratch_address(desc->device, &p->scratch);
        if (e != hipSuccess) {
            delete p;
            return hip_fail(e, "hipGetSymbolAddress(decode scratch)");
        }
        const int64_t ncnt = static_cast<int64_t>(kMaxDecodeBatch) * 16;
        if (hipMalloc(&p->counters, ncnt * sizeof(int32_t)) != hipSuccess) {
            delete p;
            return fail(KV_ERR_OOM, "counter allocation failed");
        }
        e = hck::launch_fill_i32(p->counters, ncnt, 0, static_cast<hipStream_t>(stream));
        if (e != hipSuccess) {
            delete p;
            return hip_fail(e, "counter fill");
        }
        e = hck::launch_fill_i32(page_table,
                                 static_cast<int64_t>(desc->max_sessions) * desc->max_pages_per_session,
                                 -1, static_cast<hipStream_t>(stream));
        if (e != hipSuccess) {
            delete p;
            return hip_fail(e, "page-table fill");
        }
    }
    p->st.free_hot_pages = desc->num_hot_pages;
    p->st.free_cold_pages = desc->num_cold_pages;
    *out = p;
    return KV_OK;
}

void kv_pool_destroy(kv_pool* pool) { delete pool; }

int kv_pool_stats(const kv_pool* pool, kv_pool_stats_t* out) {
    if (!pool || !out) return fail(KV_ERR_INVALID, "NULL argument");
    *out = pool->st;
    out->free_hot_pages = pool->hot_free.free_count();
    out->free_cold_pages = pool->cold_free.free_count();
    int32_t a = 0, p = 0;
    int64_t cold_active = 0;
    for (const auto& s : pool->sessions) {
        a += s.state == KV_SESSION_ACTIVE;
        p += s.state == KV_SESSION_PAUSED;
        if (s.state == KV_SESSION_ACTIVE)
            for (int32_t h : s.hot) cold_active += h < 0;
    }
    out->cold_active_pages = cold_active;
    out->active_sessions = a;
    out->paused_sessions = p;
    return KV_OK;
}

int kv_session_create(kv_pool* pool, int32_t seq_len, const int32_t* hot_pages, kv_stream_t stream,
                      int32_t* sid_out) {
    if (!pool || !sid_out) return fail(KV_ERR_INVALID, "NULL argument");
    if (seq_len < 0) return fail(KV_ERR_INVALID, "negative length");
    const int32_t n = pages_of(seq_len);
    if (n > pool->d.max_pages_per_session)
        return fail(KV_ERR_INVALID, "%d pages exceed the row stride %d", n,
                    pool->d.max_pages_per_session);
    const int32_t sid = pool->new_sid();
    if (sid < 0) return fail(KV_ERR_INVALID, "no free session slot");
    Alloc a;
    if (hot_pages) {
        a.pages.assign(hot_pages, hot_pages + n);
        std::vector<int32_t> sorted = a.pages;
        std::sort(sorted.begin(), sorted.end());
        if (std::adjacent_find(sorted.begin(), sorted.end()) != sorted.end())
            return fail(KV_ERR_INVALID, "duplicate hot page");
        for (int32_t p : a.pages)
            if (p < 0 || p >= pool->d.num_hot_pages || !pool->hot_free.is_free(p))
                return fail(KV_ERR_INVALID, "hot page %d is not free", p);
    } else {
        int rc = pool->plan_alloc(n, {}, a);
        if (rc) return rc;
    }
    const std::vector<int32_t> entries = kv_pool::new_entries(a);
    if (!pool->meta && n > 0) {
        DeviceGuard g(pool->d.device);
        hipStream_t s = pool->strm(stream);
        int rc = pool->order_after_frees(s);
        if (!rc) rc = pool->submit_victims(a, s);
        if (!rc) rc = pool->submit_row_at(sid, 0, entries.data(), n, s);
        if (rc) return rc;
    }
    pool->commit_victims(a);
    pool->commit_spill(a);
    for (int32_t p : a.pages) pool->hot_free.take(p);
    const size_t nh = a.pages.size(), ns = a.spill_cold.size();
    Session& ss = pool->sessions[sid];
    ss = Session();
    ss.state = KV_SESSION_ACTIVE;
    ss.seq_len = seq_len;
    ss.hot = a.pages;
    ss.hot.resize(nh + ns, -1);
    ss.cold.assign(nh, -1);
    ss.cold.insert(ss.cold.end(), a.spill_cold.begin(), a.spill_cold.end());
    ss.spilled.assign(nh, 0);
    ss.spilled.resize(nh + ns, 1);
    *sid_out = sid;
    return KV_OK;
}

int kv_session_extend(kv_pool* pool, int32_t sid, int32_t new_seq_len, kv_stream_t stream) {
    if (!pool) return fail(KV_ERR_INVALID, "NULL pool");
    Session* s = pool->session(sid);
    if (!s) return fail(KV_ERR_INVALID, "bad session id %d", sid);
    if (s->state != KV_SESSION_ACTIVE) return fail(KV_ERR_STATE, "session %d is not active", sid);
    if (new_seq_len < s->seq_len) return fail(KV_ERR_INVALID, "a session only grows");
    const int32_t n_old = static_cast<int32_t>(s->hot.size());
    const int32_t n_new = pages_of(new_seq_len);
    if (n_new > pool->d.max_pages_per_session)
        return fail(KV_ERR_INVALID, "%d pages exceed the row stride %d", n_new,
                    pool->d.max_pages_per_session);
    // The new tokens go into the partially filled tail page, if any: extending
    // counts as writing it (so appends resolved on the device need no
    // bookkeeping), and a spilled tail page shared with another session cannot
    // be written.
    const int32_t tail = (new_seq_len > s->seq_len && s->seq_len % KV_PAGE_TOKENS) ? s->seq_len / KV_PAGE_TOKENS : -1;
    if (tail >= 0 && s->hot[tail] < 0 && pool->cold_ref[s->cold[tail]] > 1)
        return fail(KV_ERR_STATE, "tail page %d is spilled to a cold page shared with another session", tail);
    Alloc a;
    int rc = pool->plan_alloc(std::max(n_new - n_old, 0), {}, a);
    if (rc) return rc;
    const std::vector<int32_t> entries = kv_pool::new_entries(a);
    if (!pool->meta && n_new > n_old) {
        DeviceGuard g(pool->d.device);
        hipStream_t st = pool->strm(stream);
        rc = pool->order_after_frees(st);
        if (!rc) rc = pool->submit_victims(a, st);
        if (!rc) rc = pool->submit_row_at(sid, n_old, entries.data(), n_new - n_old, st);
        if (rc) return rc;
    }
    pool->commit_victims(a);
    pool->commit_spill(a);
    for (int32_t p : a.pages) pool->hot_free.take(p);
    if (tail >= 0 && s->hot[tail] >= 0 && s->cold[tail] >= 0) {  // its cold copy goes stale
        pool->release_cold(s->cold[tail]);
        s->cold[tail] = -1;
    }
    s->hot.insert(s->hot.end(), a.pages.begin(), a.pages.end());
    s->hot.resize(n_new, -1);
    s->cold.resize(n_old + a.pages.size(), -1);
    s->cold.insert(s->cold.end(), a.spill_cold.begin(), a.spill_cold.end());
    s->spilled.resize(n_old + a.pages.size(), 0);
    s->spilled.resize(n_new, 1);
    s->seq_len = new_seq_len;
    return KV_OK;
}

int kv_session_pause(kv_pool* pool, int32_t sid) {
    if (!pool) return fail(KV_ERR_INVALID, "NULL pool");
    Session* s = pool->session(sid);
    if (!s) return fail(KV_ERR_INVALID, "bad session id %d", sid);
    if (s->state != KV_SESSION_ACTIVE) return fail(KV_ERR_STATE, "session %d is not active", sid);
    s->state = KV_SESSION_PAUSED;
    s->stamp = ++pool->clock;
    if (kv_pool::has_resident(*s)) pool->lru[s->stamp] = sid;
    return KV_OK;
}

int kv_evict_pages(kv_pool* pool, int32_t n, kv_stream_t stream, int32_t* evicted) {
    if (!pool || n < 0) return fail(KV_ERR_INVALID, "bad arguments");
    Alloc a;
    pool->plan_lru(n, {}, a.victims);
    int rc = pool->plan_victim_cold(a);
    if (rc) return rc;
    if (!pool->meta && !a.victims.empty()) {
        DeviceGuard g(pool->d.device);
        rc = pool->submit_victims(a, pool->strm(stream));
        if (rc) return rc;
    }
    pool->commit_victims(a);
    if (evicted) *evicted = static_cast<int32_t>(a.victims.size());
    return KV_OK;
}

int kv_session_import_cold(kv_pool* pool, int32_t seq_len, const int32_t* cold_pages,
                           int32_t* sid_out) {
    if (!pool || !sid_out || (seq_len > 0 && !cold_pages)) return fail(KV_ERR_INVALID, "NULL argument");
    if (seq_len < 0) return fail(KV_ERR_INVALID, "negative length");
    const int32_t n = pages_of(seq_len);
    if (n > pool->d.max_pages_per_session) return fail(KV_ERR_INVALID, "too many pages");
    std::vector<int32_t> pages(cold_pages, cold_pages + n);
    std::vector<int32_t> sorted = pages;
    std::sort(sorted.begin(), sorted.end());
    if (std::adjacent_find(sorted.begin(), sorted.end()) != sorted.end())
        return fail(KV_ERR_INVALID, "duplicate cold page");
    for (int32_t p : pages)
        if (p < 0 || p >= pool->d.num_cold_pages) return fail(KV_ERR_INVALID, "bad cold page %d", p);
    const int32_t sid = pool->new_sid();
    if (sid < 0) return fail(KV_ERR_INVALID, "no free session slot");
    for (int32_t p : pages) {
        if (pool->cold_ref[p]++ == 0) pool->cold_free.take(p);
    }
    Session& ss = pool->sessions[sid];
    ss = Session();
    ss.state = KV_SESSION_PAUSED;
    ss.seq_len = seq_len;
    ss.stamp = ++pool->clock;
    ss.hot.assign(n, -1);
    ss.cold = pages;
    ss.spilled.assign(n, 0);
    *sid_out = sid;
    return KV_OK;
}

int kv_session_destroy(kv_pool* pool, int32_t sid, kv_stream_t stream) {
    if (!pool) return fail(KV_ERR_INVALID, "NULL pool");
    Session* s = pool->session(sid);
    if (!s) return fail(KV_ERR_INVALID, "bad session id %d", sid);
    if (s->state == KV_SESSION_FREE) return fail(KV_ERR_STATE, "session %d is not in use", sid);
    if (!pool->meta && kv_pool::has_row_entries(*s)) {
        DeviceGuard g(pool->d.device);
        hipStream_t st = pool->strm(stream);
        int rc = pool->clear_row(sid, static_cast<int32_t>(s->hot.size()), st);
        if (!rc) rc = pool->note_frees(st);
        if (rc) return rc;
    }
    for (int32_t p : s->hot)
        if (p >= 0) pool->hot_free.give(p);
    for (int32_t c : s->cold)
        if (c >= 0) pool->release_cold(c);
    if (s->state == KV_SESSION_PAUSED) pool->lru.erase(s->stamp);
    *s = Session();
    return KV_OK;
}

int kv_session_info(const kv_pool* pool, int32_t sid, int32_t* state, int32_t* seq_len,
                    int32_t* hot_pages, int32_t* cold_pages, int32_t cap) {
    if (!pool) return fail(KV_ERR_INVALID, "NULL pool");
    if (sid < 0 || sid >= pool->d.max_sessions) return fail(KV_ERR_INVALID, "bad session id %d", sid);
    const Session& s = pool->sessions[sid];
    if (state) *state = s.state;
    if (seq_len) *seq_len = s.seq_len;
    if (hot_pages)
        for (int32_t i = 0; i < cap && i < static_cast<int32_t>(s.hot.size()); ++i) hot_pages[i] = s.hot[i];
    if (cold_pages)
        for (int32_t i = 0; i < cap && i < static_cast<int32_t>(s.cold.size()); ++i) cold_pages[i] = s.cold[i];
    return KV_OK;
}

int kv_append_tokens(kv_pool* pool, int32_t layer, const int32_t* sids, const int32_t* positions, int32_t n,
                     const void* k, const void* v, kv_stream_t stream) {
    if (!pool) return fail(KV_ERR_INVALID, "NULL pool");
    if (layer < 0 || layer >= pool->d.num_layers) return fail(KV_ERR_INVALID, "bad layer %d", layer);
    if (n < 0 || n > kMaxDecodeBatch || (n > 0 && (!sids || !positions)))
        return fail(KV_ERR_INVALID, "bad arguments");
    if (n == 0) return KV_OK;
    std::vector<std::pair<int32_t, int32_t>> seen(static_cast<size_t>(n));
    for (int32_t i = 0; i < n; ++i) {
        const Session* s = pool->session(sids[i]);
        if (!s) return fail(KV_ERR_INVALID, "bad session id %d", sids[i]);
        if (s->state != KV_SESSION_ACTIVE) return fail(KV_ERR_STATE, "session %d is not active", sids[i]);
        if (positions[i] < 0 || positions[i] >= s->seq_len)
            return fail(KV_ERR_INVALID, "token %d outside session %d", positions[i], sids[i]);
        const int32_t p = positions[i] / KV_PAGE_TOKENS;
        if (s->hot[p] < 0 && pool->cold_ref[s->cold[p]] > 1)
            return fail(KV_ERR_STATE, "page %d is spilled to a cold page shared with another session", p);
        seen[i] = {sids[i], positions[i]};
    }
    std::sort(seen.begin(), seen.end());
    for (int32_t i = 1; i < n; ++i)
        if (seen[i] == seen[i - 1]) return fail(KV_ERR_INVALID, "token %d of session %d given twice",
                                                seen[i].second, seen[i].first);
    if (!pool->meta) {
        if (!k || !v) return fail(KV_ERR_INVALID, "NULL k or v");
        DeviceGuard g(pool->d.device);
        hipStream_t st = pool->strm(stream);
        // short lists travel in the kernel arguments, longer ones through a staging slot
        hck::AppendArgs a;
        StagingSlot* slot = nullptr;
        hck::AppendEntry* ent = a.inline_entries;
        if (n > hck::kAppendInline) {
            int rc = pool->acquire_slot(&slot);
            if (rc) return rc;
            ent = static_cast<hck::AppendEntry*>(slot->host);
        }
        for (int32_t i = 0; i < n; ++i) {
            const Session& s = pool->sessions[sids[i]];
            const int32_t p = positions[i] / KV_PAGE_TOKENS;
            ent[i].page = s.hot[p] >= 0 ? s.hot[p] : (s.cold[p] | KV_PAGE_COLD);
            ent[i].slot = positions[i] % KV_PAGE_TOKENS;
        }
        a.entries = nullptr;
        if (slot) {
            hipError_t e = hipMemcpyAsync(slot->dev, slot->host, static_cast<size_t>(n) * sizeof(hck::AppendEntry),
                                          hipMemcpyHostToDevice, st);
            if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync(append list)");
            a.entries = static_cast<const hck::AppendEntry*>(slot->dev);
        }
        a.hot = pool->hot_geom;
        a.cold = pool->cold_geom;
        a.n = n;
        a.num_kv_heads = pool->d.num_kv_heads;
        a.head_dim = pool->d.head_dim;
        a.dtype = pool->d.dtype;
        a.layer = layer;
        a.k = k;
        a.v = v;
        hipError_t e = hck::launch_append_tokens(a, st);
        if (e != hipSuccess) return hip_fail(e, "append_tokens launch");
        if (slot) {
            e = hipEventRecord(slot->done, st);
            if (e != hipSuccess) return hip_fail(e, "hipEventRecord(staging)");
            slot->pending = true;
        }
    }
    for (int32_t i = 0; i < n; ++i) {      // a written hot page loses its cold copy
        Session& s = pool->sessions[sids[i]];
        const int32_t p = positions[i] / KV_PAGE_TOKENS;
        if (s.hot[p] >= 0 && s.cold[p] >= 0) {
            pool->release_cold(s.cold[p]);
            s.cold[p] = -1;
        }
    }
    return KV_OK;
}

int kv_write_tokens_layers(kv_pool* pool, int32_t sid, int32_t layer_begin, int32_t num_layers,
                           int32_t tok_begin, int32_t n_tok, const void* k, const void* v, kv_stream_t stream) {
    if (!pool) return fail(KV_ERR_INVALID, "NULL pool");
    Session* s = pool->session(sid);
    if (!s) return fail(KV_ERR_INVALID, "bad session id %d", sid);
    if (s->state != KV_SESSION_ACTIVE) return fail(KV_ERR_STATE, "session %d is not active", sid);
    if (layer_begin < 0 || num_layers < 1 || layer_begin + static_cast<int64_t>(num_layers) > pool->d.num_layers)
        return fail(KV_ERR_INVALID, "layers [%d, %d) outside the pool's %d", layer_begin, layer_begin + num_layers,
                    pool->d.num_layers);
    if (tok_begin < 0 || n_tok < 0 || static_cast<int64_t>(tok_begin) + n_tok > s->seq_len)
        return fail(KV_ERR_INVALID, "token range outside the session");
    if (n_tok == 0) return KV_OK;
    const int32_t first = tok_begin / KV_PAGE_TOKENS, last = (tok_begin + n_tok - 1) / KV_PAGE_TOKENS;
    for (int32_t i = first; i <= last; ++i)
        if (s->hot[i] < 0 && pool->cold_ref[s->cold[i]] > 1)
            return fail(KV_ERR_STATE, "page %d is spilled to a cold page shared with another session", i);
    if (!pool->meta) {
        if (!k || !v) return fail(KV_ERR_INVALID, "NULL k or v");
        if ((reinterpret_cast<uintptr_t>(k) | reinterpret_cast<uintptr_t>(v)) & 15)
            return fail(KV_ERR_INVALID, "k and v must be 16-byte aligned");
        DeviceGuard g(pool->d.device);
        hck::WriteArgs a;
        a.hot = pool->hot_geom;
        a.cold = pool->cold_geom;
        a.row = pool->pt + static_cast<int64_t>(sid) * pool->d.max_pages_per_session;
        a.num_kv_heads = pool->d.num_kv_heads;
        a.head_dim = pool->d.head_dim;
        a.dtype = pool->d.dtype;
        a.layer = layer_begin;
        a.num_layers = num_layers;
        a.tok_begin = tok_begin;
        a.n_tok = n_tok;
        a.k = k;
        a.v = v;
        hipError_t e = hck::launch_write_tokens(a, pool->strm(stream));
        if (e != hipSuccess) return hip_fail(e, "write_tokens launch");
    }
    for (int32_t i = first; i <= last; ++i) {
        if (s->hot[i] >= 0 && s->cold[i] >= 0) {   // a spilled page is written in place
            pool->release_cold(s->cold[i]);
            s->cold[i] = -1;
        }
    }
    return KV_OK;
}

int kv_write_tokens(kv_pool* pool, int32_t sid, int32_t layer, int32_t tok_begin, int32_t n_tok,
                    const void* k, const void* v, kv_stream_t stream) {
    if (pool && (layer < 0 || layer >= pool->d.num_layers)) return fail(KV_ERR_INVALID, "bad layer %d", layer);
    return kv_write_tokens_layers(pool, sid, layer, 1, tok_begin, n_tok, k, v, stream);
}

int kv_append_tokens_table(kv_pool* pool, int32_t layer_begin, int32_t num_layers, const int32_t* table,
                           int64_t pt_stride, int32_t table_rows, const int32_t* rows, const int32_t* positions,
                           int32_t n, const void* k, const void* v, kv_stream_t stream) {
    if (!pool) return fail(KV_ERR_INVALID, "NULL pool");
    if (pool->meta) return fail(KV_ERR_INVALID, "metadata-only pool has no pages");
    if (layer_begin < 0 || num_layers < 1 || layer_begin + static_cast<int64_t>(num_layers) > pool->d.num_layers)
        return fail(KV_ERR_INVALID, "layers [%d, %d) outside the pool's %d", layer_begin, layer_begin + num_layers,
                    pool->d.num_layers);
    if (n < 0 || n > kMaxDecodeBatch) return fail(KV_ERR_INVALID, "n %d outside [0, %d]", n, kMaxDecodeBatch);
    if (n == 0) return KV_OK;
    if (!table || !rows || !positions || !k || !v) return fail(KV_ERR_INVALID, "NULL buffer");
    if (pt_stride < 1 || table_rows < 0 || static_cast<int64_t>(table_rows) * pt_stride >= (int64_t(1) << 31))
        return fail(KV_ERR_INVALID, "bad page-table shape");
    if ((reinterpret_cast<uintptr_t>(k) | reinterpret_cast<uintptr_t>(v)) & 15)
        return fail(KV_ERR_INVALID, "k and v must be 16-byte aligned");
    DeviceGuard g(pool->d.device);
    hck::AppendTableArgs a;
    a.hot = pool->hot_geom;
    a.cold = pool->cold_geom;
    a.num_hot = pool->d.num_hot_pages;
    a.num_cold = pool->cold ? pool->d.num_cold_pages : 0;
    a.table = table;
    a.pt_stride = pt_stride;
    a.table_rows = table_rows;
    a.rows = rows;
    a.positions = positions;
    a.n = n;
    a.num_kv_heads = pool->d.num_kv_heads;
    a.head_dim = pool->d.head_dim;
    a.dtype = pool->d.dtype;
    a.layer = layer_begin;
    a.num_layers = num_layers;
    a.k = k;
    a.v = v;
    hipError_t e = hck::launch_append_table(a, pool->strm(stream));
    if (e != hipSuccess) return hip_fail(e, "append_table launch");
    return KV_OK;
}

int kv_fill_synthetic_pages(kv_pool* pool, int32_t sid, int32_t gen_sid, uint64_t seed,
                            float value_mult, int32_t first_page, int32_t num_pages,
                            kv_stream_t stream) {
    if (!pool) return fail(KV_ERR_INVALID, "NULL pool");
    if (pool->meta) return fail(KV_ERR_INVALID, "metadata-only pool has no pages");
    Session* s = pool->session(sid);
    if (!s) return fail(KV_ERR_INVALID, "bad session id %d", sid);
    if (s->state != KV_SESSION_ACTIVE) return fail(KV_ERR_STATE, "session %d is not active", sid);
    if (gen_sid < 0 || gen_sid >= (1 << 20)) return fail(KV_ERR_INVALID, "gen_sid out of range");
    const int64_t have = static_cast<int64_t>(s->hot.size());
    if (first_page < 0 || num_pages < 0 || first_page + static_cast<int64_t>(num_pages) > have)
        return fail(KV_ERR_INVALID, "pages [%d, %d) outside the session's %lld", first_page,
                    first_page + num_pages, static_cast<long long>(have));
    if (num_pages == 0) return KV_OK;
    for (int32_t i = first_page; i < first_page + num_pages; ++i)
        if (s->hot[i] < 0 && pool->cold_ref[s->cold[i]] > 1)
            return fail(KV_ERR_STATE, "page %d is spilled to a cold page shared with another session", i);
    DeviceGuard g(pool->d.device);
    hck::SynthArgs a;
    a.hot = pool->hot_geom;
    a.cold = pool->cold_geom;
    a.slice_bytes = pool->slice_bytes;
    a.row = pool->pt + static_cast<int64_t>(sid) * pool->d.max_pages_per_session;
    a.first_page = first_page;
    a.num_pages = num_pages;
    a.num_layers = pool->d.num_layers;
    a.num_kv_heads = pool->d.num_kv_heads;
    a.head_dim = pool->d.head_dim;
    a.dtype = pool->d.dtype;
    a.gen_sid = gen_sid;
    a.seed = seed;
    a.value_mult = value_mult;
    hipError_t e = hck::launch_fill_synthetic(a, pool->strm(stream));
    if (e != hipSuccess) return hip_fail(e, "fill_synthetic launch");
    for (int32_t i = first_page; i < first_page + num_pages; ++i) {
        if (s->hot[i] >= 0 && s->cold[i] >= 0) {   // a spilled page is written in place
            pool->release_cold(s->cold[i]);
            s->cold[i] = -1;
        }
    }
    return KV_OK;
}

int kv_fill_synthetic(kv_pool* pool, int32_t sid, int32_t gen_sid, uint64_t seed, float value_mult,
                      kv_stream_t stream) {
    if (!pool) return fail(KV_ERR_INVALID, "NULL pool");
    Session* s = pool->session(sid);
    if (!s) return fail(KV_ERR_INVALID, "bad session id %d", sid);
    return kv_fill_synthetic_pages(pool, sid, gen_sid, seed, value_mult, 0,
                                   static_cast<int32_t>(s->hot.size()), stream);
}

int kv_pool_set_spill(kv_pool* pool, int32_t enable) {
    if (!pool || (enable != 0 && enable != 1)) return fail(KV_ERR_INVALID, "bad arguments");
    if (!enable) {
        // Without spill, decode reads the pool's rows with the plain kernel, for
        // which a cold-tagged entry is an invalid id: refuse while rows name
        // spilled pages (promote them, or evict their sessions, first).
        for (size_t sid = 0; sid < pool->sessions.size(); ++sid)
            for (uint8_t sp : pool->sessions[sid].spilled)
                if (sp)
                    return fail(KV_ERR_STATE, "session %zu still has pages in the cold tier", sid);
    }
    pool->spill = enable != 0;
    return KV_OK;
}

int kv_promote_pages(kv_pool* pool, int32_t n, kv_stream_t stream, int32_t* promoted) {
    if (!pool || n < 0) return fail(KV_ERR_INVALID, "bad arguments");
    // spilled pages of active sessions: session id order, logical page order
    std::vector<Victim> want;
    for (int32_t sid = 0; sid < pool->d.max_sessions && static_cast<int32_t>(want.size()) < n; ++sid) {
        const Session& s = pool->sessions[sid];
        if (s.state != KV_SESSION_ACTIVE) continue;
        for (size_t i = 0; i < s.hot.size() && static_cast<int32_t>(want.size()) < n; ++i)
            if (s.hot[i] < 0) want.push_back(Victim{sid, static_cast<int32_t>(i)});
    }
    Alloc a;
    int rc = pool->plan_alloc(static_cast<int64_t>(want.size()), {}, a, /*fresh_spill=*/false,
                              /*allow_spill=*/true);
    if (rc) return rc;
    if (!pool->meta && !a.pages.empty()) {
        DeviceGuard g(pool->d.device);
        hipStream_t st = pool->strm(stream);
        // Two phases: the copies, then (stream-ordered after them) the row
        // entries.  A decode running meanwhile on another stream reads either
        // the cold id (the cold copy stays valid) or a fully copied hot page.
        std::vector<hck::CopyEntry> copies, writes;
        for (size_t k = 0; k < a.pages.size(); ++k) {
            const Victim& w = want[k];
            copies.push_back(hck::CopyEntry{pool->sessions[w.sid].cold[w.page], a.pages[k], -1, 0});
            writes.push_back(hck::CopyEntry{-1, -1, w.sid * pool->d.max_pages_per_session + w.page,
                                            a.pages[k]});
        }
        rc = pool->order_after_frees(st);
        if (!rc) rc = pool->submit_victims(a, st);
        if (!rc) rc = pool->submit_copies(true, copies, st, KV_KERNEL_PAGE_COPY);
        if (!rc) rc = pool->submit_table_writes(writes, st);
        if (rc) return rc;
    }
    pool->commit_victims(a);
    for (size_t k = 0; k < a.pages.size(); ++k) {
        Session& s = pool->sessions[want[k].sid];
        s.hot[want[k].page] = a.pages[k];
        s.spilled[want[k].page] = 0;
        pool->hot_free.take(a.pages[k]);
    }
    const int64_t m = static_cast<int64_t>(a.pages.size());
    pool->st.promoted_pages += m;
    pool->st.pages_to_hot += m;
    pool->st.bytes_to_hot += m * pool->page_bytes;
    if (promoted) *promoted = static_cast<int32_t>(m);
    return KV_OK;
}

int kv_evict_sessions(kv_pool* pool, const int32_t* sids, int32_t n, kv_stream_t stream) {
    if (!pool || (n > 0 && !sids) || n < 0) return fail(KV_ERR_INVALID, "bad arguments");
    if (n == 0) return KV_OK;
    std::vector<int32_t> ids(sids, sids + n);
    {
        std::vector<int32_t> sorted = ids;
        std::sort(sorted.begin(), sorted.end());
        if (std::adjacent_find(sorted.begin(), sorted.end()) != sorted.end())
            return fail(KV_ERR_INVALID, "duplicate session in batch");
    }
    int64_t dirty = 0;
    for (int32_t sid : ids) {
        Session* s = pool->session(sid);
        if (!s) return fail(KV_ERR_INVALID, "bad session id %d", sid);
        if (s->state != KV_SESSION_ACTIVE) return fail(KV_ERR_STATE, "session %d is not active", sid);
        for (int32_t c : s->cold) dirty += c < 0;
    }
    if (dirty > pool->cold_free.free_count())
        return fail(KV_ERR_NO_COLD_PAGES, "need %lld cold pages, %d free", static_cast<long long>(dirty),
                    pool->cold_free.free_count());
    // cold pages for the dirty pages, lowest first, in argument and logical-page order
    std::vector<int32_t> dst;
    pool->cold_free.lowest(static_cast<int32_t>(dirty), dst);
    if (!pool->meta) {
        DeviceGuard g(pool->d.device);
        hipStream_t st = pool->strm(stream);
        std::vector<hck::CopyEntry> entries;
        size_t k = 0;
        for (int32_t sid : ids) {
            const Session& s = pool->sessions[sid];
            const int32_t row = sid * pool->d.max_pages_per_session;
            for (size_t i = 0; i < s.hot.size(); ++i) {
                const bool copy = s.cold[i] < 0;
                entries.push_back(hck::CopyEntry{copy ? s.hot[i] : -1, copy ? dst[k] : -1,
                                                 row + static_cast<int32_t>(i), -1});
                k += copy;
            }
        }
        int rc = pool->submit_copies(false, entries, st, KV_KERNEL_EVICT_COPY);
        if (!rc) rc = pool->note_frees(st);
        if (rc) return rc;
    }
    size_t k = 0;
    for (int32_t sid : ids) {
        Session& s = pool->sessions[sid];
        int64_t written = 0;
        for (size_t i = 0; i < s.cold.size(); ++i) {
            if (s.cold[i] < 0) {
                pool->cold_free.take(dst[k]);
                pool->cold_ref[dst[k]] = 1;
                s.cold[i] = dst[k++];
                ++written;
            }
            if (s.hot[i] >= 0) pool->hot_free.give(s.hot[i]);
            s.hot[i] = -1;
            s.spilled[i] = 0;
        }
        s.state = KV_SESSION_PAUSED;
        s.stamp = ++pool->clock;
        pool->st.pages_to_cold += written;
        pool->st.bytes_to_cold += written * pool->page_bytes;
        pool->st.evicts += 1;
    }
    return KV_OK;
}

int kv_evict_session(kv_pool* pool, int32_t sid, kv_stream_t stream) {
    return kv_evict_sessions(pool, &sid, 1, stream);
}

int kv_resume_sessions(kv_pool* pool, const int32_t* sids, int32_t n, kv_stream_t stream) {
    if (!pool || (n > 0 && !sids) || n < 0) return fail(KV_ERR_INVALID, "bad arguments");
    if (n == 0) return KV_OK;
    std::vector<int32_t> ids(sids, sids + n);
    {
        std::vector<int32_t> sorted = ids;
        std::sort(sorted.begin(), sorted.end());
        if (std::adjacent_find(sorted.begin(), sorted.end()) != sorted.end())
            return fail(KV_ERR_INVALID, "duplicate session in batch");
    }
    int64_t need = 0;
    for (int32_t sid : ids) {
        Session* s = pool->session(sid);
        if (!s) return fail(KV_ERR_INVALID, "bad session id %d", sid);
        if (s->state != KV_SESSION_PAUSED) return fail(KV_ERR_STATE, "session %d is not paused", sid);
        for (int32_t p : s->hot) need += p < 0;
    }
    // the sessions being resumed keep their resident pages: never evict those;
    // with spill, pages that find no hot page stay in the cold tier
    Alloc a;
    int rc = pool->plan_alloc(need, ids, a, /*fresh_spill=*/false);
    if (rc) return rc;
    if (!pool->meta) {
        DeviceGuard g(pool->d.device);
        hipStream_t st = pool->strm(stream);
        std::vector<hck::CopyEntry> entries;
        size_t k = 0;
        for (int32_t sid : ids) {
            const Session& s = pool->sessions[sid];
            const int32_t row = sid * pool->d.max_pages_per_session;
            for (size_t i = 0; i < s.hot.size(); ++i) {
                if (s.hot[i] < 0 && k < a.pages.size()) {
                    entries.push_back(hck::CopyEntry{s.cold[i], a.pages[k], row + static_cast<int32_t>(i),
                                                     a.pages[k]});
                    ++k;
                } else if (s.hot[i] < 0) {
                    entries.push_back(hck::CopyEntry{-1, -1, row + static_cast<int32_t>(i),
                                                     s.cold[i] | KV_PAGE_COLD});
                } else {
                    entries.push_back(hck::CopyEntry{-1, -1, row + static_cast<int32_t>(i), s.hot[i]});
                }
            }
        }
        rc = pool->order_after_frees(st);
        if (!rc) rc = pool->submit_victims(a, st);
        if (!rc) rc = pool->submit_copies(true, entries, st, KV_KERNEL_PAGE_COPY);
        if (rc) return rc;
    }
    pool->commit_victims(a);
    size_t k = 0;
    for (int32_t sid : ids) {
        Session& s = pool->sessions[sid];
        int64_t fetched = 0, resident = 0;
        for (size_t i = 0; i < s.hot.size(); ++i) {
            if (s.hot[i] >= 0) {
                ++resident;
            } else if (k < a.pages.size()) {
                s.hot[i] = a.pages[k++];
                s.spilled[i] = 0;
                pool->hot_free.take(s.hot[i]);
                ++fetched;
            } else {
                s.spilled[i] = 1;
                pool->st.spilled_pages += 1;
            }
        }
        pool->lru.erase(s.stamp);
        s.state = KV_SESSION_ACTIVE;
        pool->st.pages_to_hot += fetched;
        pool->st.bytes_to_hot += fetched * pool->page_bytes;
        pool->st.resume_pages_resident += resident;
        pool->st.resume_pages_total += static_cast<int64_t>(s.hot.size());
        pool->st.resumes += 1;
    }
    return KV_OK;
}

int kv_resume_sessions_lazy(kv_pool* pool, const int32_t* sids, int32_t n, kv_stream_t stream) {
    if (!pool || (n > 0 && !sids) || n < 0) return fail(KV_ERR_INVALID, "bad arguments");
    if (!pool->spill) return fail(KV_ERR_INVALID, "lazy resume needs spill on");
    if (n == 0) return KV_OK;
    std::vector<int32_t> ids(sids, sids + n);
    {
        std::vector<int32_t> sorted = ids;
        std::sort(sorted.begin(), sorted.end());
        if (std::adjacent_find(sorted.begin(), sorted.end()) != sorted.end())
            return fail(KV_ERR_INVALID, "duplicate session in batch");
    }
    for (int32_t sid : ids) {
        Session* s = pool->session(sid);
        if (!s) return fail(KV_ERR_INVALID, "bad session id %d", sid);
        if (s->state != KV_SESSION_PAUSED) return fail(KV_ERR_STATE, "session %d is not paused", sid);
    }
    if (!pool->meta) {
        DeviceGuard g(pool->d.device);
        hipStream_t st = pool->strm(stream);
        for (int32_t sid : ids) {
            const Session& s = pool->sessions[sid];
            std::vector<int32_t> row(s.hot.size());
            for (size_t i = 0; i < s.hot.size(); ++i)
                row[i] = s.hot[i] >= 0 ? s.hot[i] : (s.cold[i] | KV_PAGE_COLD);
            int rc = pool->submit_row_at(sid, 0, row.data(), static_cast<int32_t>(row.size()), st);
            if (rc) return rc;
        }
    }
    for (int32_t sid : ids) {
        Session& s = pool->sessions[sid];
        int64_t resident = 0;
        for (size_t i = 0; i < s.hot.size(); ++i) {
            if (s.hot[i] >= 0) {
                ++resident;
            } else {
                s.spilled[i] = 1;
                pool->st.spilled_pages += 1;
            }
        }
        pool->lru.erase(s.stamp);
        s.state = KV_SESSION_ACTIVE;
        pool->st.resume_pages_resident += resident;
        pool->st.resume_pages_total += static_cast<int64_t>(s.hot.size());
        pool->st.resumes += 1;
    }
    return KV_OK;
}

int kv_resume_session(kv_pool* pool, int32_t sid, kv_stream_t stream) {
    return kv_resume_sessions(pool, &sid, 1, stream);
}

int32_t paged_decode_waves(const kv_pool* pool) {
    if (!pool || pool->meta) return 0;
    DeviceGuard g(pool->d.device);
    return pool->decode_waves();
}

int kv_pool_set_copy_blocks(kv_pool* pool, int32_t blocks) {
    if (!pool || blocks < 0) return fail(KV_ERR_INVALID, "bad arguments");
    pool->copy_blocks = blocks;
    return KV_OK;
}

int kv_pool_set_decode_combine(kv_pool* pool, int32_t mode) {
    if (!pool || (mode != KV_COMBINE_SEPARATE && mode != KV_COMBINE_FUSED))
        return fail(KV_ERR_INVALID, "bad arguments");
    pool->combine_mode = mode;
    return KV_OK;
}

int kv_pool_set_host_copy(kv_pool* pool, int32_t mode) {
    if (!pool || (mode != KV_HOST_COPY_DMA && mode != KV_HOST_COPY_KERNEL))
        return fail(KV_ERR_INVALID, "bad arguments");
    pool->host_copy = mode;
    return KV_OK;
}

int kv_pool_set_decode_compute(kv_pool* pool, int32_t mode) {
    if (!pool || (mode != KV_DECODE_MATRIX && mode != KV_DECODE_VECTOR))
        return fail(KV_ERR_INVALID, "bad arguments");
    pool->compute_mode = mode;
    return KV_OK;
}

int kv_pool_set_decode_waves(kv_pool* pool, int32_t waves) {
    if (!pool || waves < 0) return fail(KV_ERR_INVALID, "bad arguments");
    pool->waves_override = waves;
    return KV_OK;
}

size_t paged_decode_workspace_bytes(const kv_pool* pool, int32_t batch, int32_t num_q_heads) {
    if (!pool || pool->meta || batch < 0 || num_q_heads <= 0 || num_q_heads % pool->d.num_kv_heads)
        return 0;
    const int32_t group = num_q_heads / pool->d.num_kv_heads;
    DeviceGuard g(pool->d.device);
    const int32_t waves = pool->decode_waves();
    const int64_t slots = static_cast<int64_t>(waves) + static_cast<int64_t>(batch) * pool->d.num_kv_heads;
    return hck::decode_workspace_bytes(slots, group, pool->d.head_dim, batch, waves);
}

int paged_decode_attention(kv_pool* pool, int32_t layer, const void* q, const int32_t* page_table,
                           int64_t pt_stride, const int32_t* seq_lens, int32_t batch,
                           int32_t num_q_heads, float scale, void* out, void* workspace,
                           size_t ws_bytes, kv_stream_t stream) {
    return hck::decode_impl(pool, layer, q, page_table, pt_stride, seq_lens, batch, num_q_heads, scale,
                            out, workspace, ws_bytes, stream, /*no_alloc=*/false);
}

int paged_decode_attention_append(kv_pool* pool, int32_t layer, const void* q, const void* k_new,
                                  const void* v_new, const int32_t* page_table, int64_t pt_stride,
                                  const int32_t* seq_lens, int32_t batch, int32_t num_q_heads, float scale,
                                  void* out, void* workspace, size_t ws_bytes, kv_stream_t stream) {
    if (!k_new || !v_new) return fail(KV_ERR_INVALID, "NULL k_new or v_new");
    return hck::decode_impl(pool, layer, q, page_table, pt_stride, seq_lens, batch, num_q_heads, scale,
                            out, workspace, ws_bytes, stream, /*no_alloc=*/false, k_new, v_new);
}

}  // extern "C"

namespace hck {

int decode_impl(kv_pool* pool, int32_t layer, const void* q, const int32_t* page_table, int64_t pt_stride,
                const int32_t* seq_lens, int32_t batch, int32_t num_q_heads, float scale, void* out,
                void* workspace, size_t ws_bytes, kv_stream_t stream, bool no_alloc, const void* k_new,
                const void* v_new) {
    if (!pool) return fail(KV_ERR_INVALID, "NULL pool");
    if (pool->meta) return fail(KV_ERR_INVALID, "metadata-only pool cannot decode");
    if (layer < 0 || layer >= pool->d.num_layers) return fail(KV_ERR_INVALID, "bad layer %d", layer);
    if (batch < 0 || batch > kMaxDecodeBatch)
        return fail(KV_ERR_INVALID, "batch %d outside [0, %d]", batch, kMaxDecodeBatch);
    if (batch == 0) return KV_OK;
    if (!q || !page_table || !seq_lens || !out || !workspace) return fail(KV_ERR_INVALID, "NULL buffer");
    if (num_q_heads <= 0 || num_q_heads % pool->d.num_kv_heads)
        return fail(KV_ERR_INVALID, "query heads %d not a multiple of KV heads %d", num_q_heads,
                    pool->d.num_kv_heads);
    const int32_t group = num_q_heads / pool->d.num_kv_heads;
    if (group > 16) return fail(KV_ERR_INVALID, "more than 16 query heads per KV head");
    const bool valu = pool->compute_mode == KV_DECODE_VECTOR;
    if (valu && (pool->d.dtype != KV_DTYPE_BF16 || group > 8 || pool->combine_mode != KV_COMBINE_SEPARATE))
        return fail(KV_ERR_INVALID, "vector-ALU decode needs bf16, at most 8 query heads per KV head "
                                    "and the separate merge");
    if (pt_stride < 1 || static_cast<int64_t>(batch) * pt_stride >= (int64_t(1) << 31))
        return fail(KV_ERR_INVALID, "bad page-table stride");
    if (reinterpret_cast<uintptr_t>(workspace) & 255)
        return fail(KV_ERR_INVALID, "workspace must be 256-byte aligned");
    if ((reinterpret_cast<uintptr_t>(q) | reinterpret_cast<uintptr_t>(out)) & 15)
        return fail(KV_ERR_INVALID, "q and out must be 16-byte aligned");
    if ((k_new != nullptr) != (v_new != nullptr) ||
        ((reinterpret_cast<uintptr_t>(k_new) | reinterpret_cast<uintptr_t>(v_new)) & 15))
        return fail(KV_ERR_INVALID, "k_new and v_new: both or neither, 16-byte aligned");
    DeviceGuard g(pool->d.device);
    const int32_t waves = pool->decode_waves();
    const int64_t slots = static_cast<int64_t>(waves) + static_cast<int64_t>(batch) * pool->d.num_kv_heads;
    const size_t need = hck::decode_workspace_bytes(slots, group, pool->d.head_dim, batch, waves);
    if (ws_bytes < need) {
        if (no_alloc)
            return fail(KV_ERR_INVALID, "this batch needs %zu bytes of decode scratch; the no-allocation "
                                        "entry point has %zu (use paged_decode_attention)", need, ws_bytes);
        return fail(KV_ERR_INVALID, "workspace %zu bytes, need %zu", ws_bytes, need);
    }
    hck::DecodeArgs a;
    a.hot = hck::slice_at(pool->hot_geom, 0, layer);
    a.hot_stride = pool->hot_geom.page_stride;
    a.num_pages = pool->d.num_hot_pages;
    a.num_kv_heads = pool->d.num_kv_heads;
    a.group = group;
    a.num_q_heads = num_q_heads;
    a.q = q;
    a.page_table = page_table;
    a.pt_stride = pt_stride;
    a.seq_lens = seq_lens;
    a.batch = batch;
    a.waves = waves;
    a.group_waves = hck::decode_group_waves(pool->d.num_kv_heads, waves);
    a.scale_log2 = scale * 1.4426950408889634f;
    a.part_o = static_cast<float*>(workspace);
    a.part_ml = a.part_o + slots * group * pool->d.head_dim;
    a.row_pref = reinterpret_cast<int32_t*>(static_cast<char*>(workspace) +
                                            hck::decode_partials_bytes(slots, group, pool->d.head_dim));
    a.split_segs = a.row_pref + batch + 1;
    a.combine_by_worker = 0;
    a.out = out;
    a.counters = pool->counters;
    a.fused = pool->combine_mode == KV_COMBINE_FUSED ? 1 : 0;
    a.tiered = pool->tiered() ? 1 : 0;
    a.valu = valu ? 1 : 0;
    a.cold = pool->cold ? hck::slice_at(pool->cold_geom, 0, layer) : nullptr;
    a.cold_stride = pool->cold_geom.page_stride;
    a.num_cold_pages = pool->cold ? pool->d.num_cold_pages : 0;
    a.slice_bytes = pool->slice_bytes;
    a.stage = nullptr;
    a.num_stage_slots = 0;
    a.k_new = k_new;
    a.v_new = v_new;
    const int half = layer & 1;
    const bool staged = pool->stage_slots > 0 && !pool->plan.empty() && pool->half_layer[half] == layer;
    if (staged && k_new)
        return fail(KV_ERR_INVALID, "the fused append writes pages, not staged copies: no staged layer");
    if (staged) {
        a.stage = pool->stage + static_cast<int64_t>(half) * pool->stage_slots * pool->slice_bytes;
        a.num_stage_slots = static_cast<int32_t>(pool->plan.size());
    }
    hipStream_t st = pool->strm(stream);
    // Under stream capture (a HIP graph of decode steps) the call launches its
    // two kernels only: no pool events, which belong to eager cross-stream use.
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    hipError_t ce = hipStreamIsCapturing(st, &cap);
    if (ce != hipSuccess) return hip_fail(ce, "hipStreamIsCapturing");
    const bool capturing = cap != hipStreamCaptureStatusNone;
    if (capturing && (a.fused || staged))
        return fail(KV_ERR_INVALID, "graph capture supports the separate merge without staged pages");
    // Fused-merge calls share the pool's arrival counters: order them across
    // streams.  Separate-merge calls share nothing of the pool's, so decodes on
    // different streams (say two batches on disjoint CU sets) run concurrently.
    if (a.fused && pool->decode_pending) {
        hipError_t w = hipStreamWaitEvent(st, pool->decode_event, 0);
        if (w != hipSuccess) return hip_fail(w, "hipStreamWaitEvent(decode)");
    }
    if (staged && pool->half_ready_pending[half]) {
        hipError_t w = hipStreamWaitEvent(st, pool->half_ready[half], 0);
        if (w != hipSuccess) return hip_fail(w, "hipStreamWaitEvent(staging)");
    }
    // The no-allocation entry point takes no profiling events (creating one may allocate).
    const bool prof = !capturing && !no_alloc;
    hck::LaunchEvents ev = prof ? pool->prof_events() : hck::LaunchEvents{};
    hipError_t e = hck::launch_decode_split(a, pool->d.head_dim, pool->d.dtype, st, ev);
    pool->prof_done(KV_KERNEL_DECODE_SPLIT, ev, e);
    if (e != hipSuccess) return hip_fail(e, "decode split launch");
    if (!a.fused) {
        ev = prof ? pool->prof_events() : hck::LaunchEvents{};
        e = hck::launch_decode_combine(a, pool->d.head_dim, pool->d.dtype, st, ev);
        pool->prof_done(KV_KERNEL_DECODE_COMBINE, ev, e);
        if (e != hipSuccess) return hip_fail(e, "decode combine launch");
    }
    if (capturing) return KV_OK;
    if (a.fused) {
        e = hipEventRecord(pool->decode_event, st);
        if (e != hipSuccess) return hip_fail(e, "hipEventRecord(decode)");
        pool->decode_pending = true;
    }
    if (staged) {
        e = hipEventRecord(pool->half_free[half], st);
        if (e != hipSuccess) return hip_fail(e, "hipEventRecord(staging)");
        pool->half_free_pending[half] = true;
    }
    return KV_OK;
}

int pool_scratch(kv_pool* pool, void** out) {
    *out = nullptr;
    if (!pool) return fail(KV_ERR_INVALID, "NULL pool");
    if (pool->meta || !pool->scratch) return fail(KV_ERR_INVALID, "metadata-only pool cannot decode");
    *out = pool->scratch;
    return KV_OK;
}

}  // namespace hck

extern "C" {

int kv_pool_set_staging(kv_pool* pool, void* staging, size_t bytes, int32_t* slots) {
    if (!pool || pool->meta) return fail(KV_ERR_INVALID, "no device pool");
    if (reinterpret_cast<uintptr_t>(staging) & 255) return fail(KV_ERR_INVALID, "staging must be 256-byte aligned");
    DeviceGuard g(pool->d.device);
    if (pool->decode_pending) (void)hipEventSynchronize(pool->decode_event);
    pool->free_staging_state();
    const int64_t slice = pool->slice_bytes;
    const int64_t n = staging ? static_cast<int64_t>(bytes) / (2 * slice) : 0;
    pool->stage = n > 0 ? static_cast<char*>(staging) : nullptr;
    pool->stage_slots = static_cast<int32_t>(std::min<int64_t>(n, int64_t(1) << 28));
    if (pool->stage_slots > 0) {
        for (hipEvent_t* e : {&pool->plan_ready, &pool->prefetch_done, &pool->half_ready[0],
                              &pool->half_ready[1], &pool->half_free[0], &pool->half_free[1]})
            if (!*e && hipEventCreateWithFlags(e, hipEventDisableTiming) != hipSuccess)
                return fail(KV_ERR_OOM, "event creation failed");
        const size_t eb = static_cast<size_t>(pool->stage_slots) * sizeof(hck::CopyEntry);
        if (hipMalloc(&pool->plan_dev, eb) != hipSuccess ||
            hipHostMalloc(reinterpret_cast<void**>(&pool->plan_host), eb, hipHostMallocDefault) != hipSuccess) {
            pool->stage = nullptr;
            pool->stage_slots = 0;
            return fail(KV_ERR_OOM, "staging plan allocation failed");
        }
        pool->plan_cap = pool->stage_slots;
    }
    if (slots) *slots = pool->stage_slots;
    return KV_OK;
}

int paged_decode_stage(kv_pool* pool, const int32_t* sids, int32_t n, int32_t* table,
                       kv_stream_t stream, int32_t* staged) {
    if (!pool || pool->meta) return fail(KV_ERR_INVALID, "no device pool");
    if (n < 0 || n > kMaxDecodeBatch || (n > 0 && (!sids || !table))) return fail(KV_ERR_INVALID, "bad arguments");
    for (int32_t i = 0; i < n; ++i) {
        const Session* s = pool->session(sids[i]);
        if (!s) return fail(KV_ERR_INVALID, "bad session id %d", sids[i]);
        if (s->state != KV_SESSION_ACTIVE) return fail(KV_ERR_STATE, "session %d is not active", sids[i]);
    }
    DeviceGuard g(pool->d.device);
    hipStream_t st = pool->strm(stream);
    // the previous plan's buffers must no longer be in use
    if (pool->prefetch_pending) {
        hipError_t e = hipEventSynchronize(pool->prefetch_done);
        if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize(prefetch)");
        pool->prefetch_pending = false;
    }
    if (pool->plan_ready_pending) {
        hipError_t e = hipEventSynchronize(pool->plan_ready);
        if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize(plan)");
        pool->plan_ready_pending = false;
    }
    const int32_t stride = pool->d.max_pages_per_session;
    std::vector<int32_t> rows(static_cast<size_t>(n) * stride, -1);
    std::vector<int32_t> plan;
    for (int32_t b = 0; b < n; ++b) {
        const Session& s = pool->sessions[sids[b]];
        int32_t* r = rows.data() + static_cast<size_t>(b) * stride;
        for (size_t i = 0; i < s.hot.size(); ++i) {
            if (s.hot[i] >= 0) {
                r[i] = s.hot[i];
            } else if (static_cast<int32_t>(plan.size()) < pool->stage_slots) {
                r[i] = static_cast<int32_t>(plan.size()) | KV_PAGE_STAGED;
                plan.push_back(s.cold[i]);
            } else {
                r[i] = s.cold[i] | KV_PAGE_COLD;
            }
        }
    }
    // the batch table, through the staging ring in pieces of whole rows
    const size_t row_bytes = static_cast<size_t>(stride) * sizeof(int32_t);
    const int32_t rows_per_slot = static_cast<int32_t>(kStagingBytes / row_bytes);
    for (int32_t b0 = 0; b0 < n; b0 += rows_per_slot) {
        const int32_t m = std::min(rows_per_slot, n - b0);
        StagingSlot* slot;
        int rc = pool->acquire_slot(&slot);
        if (rc) return rc;
        std::memcpy(slot->host, rows.data() + static_cast<size_t>(b0) * stride, m * row_bytes);
        hipError_t e = hipMemcpyAsync(table + static_cast<size_t>(b0) * stride, slot->host, m * row_bytes,
                                      hipMemcpyHostToDevice, st);
        if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync(batch table)");
        e = hipEventRecord(slot->done, st);
        if (e != hipSuccess) return hip_fail(e, "hipEventRecord(staging)");
        slot->pending = true;
    }
    if (!plan.empty()) {
        for (size_t k = 0; k < plan.size(); ++k)
            pool->plan_host[k] = hck::CopyEntry{plan[k], static_cast<int32_t>(k), -1, 0};
        hipError_t e = hipMemcpyAsync(pool->plan_dev, pool->plan_host, plan.size() * sizeof(hck::CopyEntry),
                                      hipMemcpyHostToDevice, st);
        if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync(staging plan)");
        e = hipEventRecord(pool->plan_ready, st);
        if (e != hipSuccess) return hip_fail(e, "hipEventRecord(plan)");
        pool->plan_ready_pending = true;
    }
    pool->plan = std::move(plan);
    pool->half_layer[0] = pool->half_layer[1] = -1;
    if (staged) *staged = static_cast<int32_t>(pool->plan.size());
    return KV_OK;
}

int paged_decode_prefetch(kv_pool* pool, int32_t layer, kv_stream_t copy_stream) {
    if (!pool || pool->meta || pool->stage_slots <= 0) return fail(KV_ERR_INVALID, "no staging buffer");
    if (layer < 0 || layer >= pool->d.num_layers) return fail(KV_ERR_INVALID, "bad layer %d", layer);
    const int half = layer & 1;
    pool->half_layer[half] = -1;
    if (pool->plan.empty()) return KV_OK;
    DeviceGuard g(pool->d.device);
    hipStream_t cs = pool->strm(copy_stream);
    hipError_t e = hipSuccess;
    if (pool->plan_ready_pending) e = hipStreamWaitEvent(cs, pool->plan_ready, 0);
    if (e == hipSuccess && pool->half_free_pending[half]) e = hipStreamWaitEvent(cs, pool->half_free[half], 0);
    if (e != hipSuccess) return hip_fail(e, "hipStreamWaitEvent(prefetch)");
    // layer `layer` of each planned cold page into its staging slot
    const hck::PoolGeom src{hck::slice_at(pool->cold_geom, 0, layer), pool->cold_geom.page_stride, 0};
    const hck::PoolGeom dst{pool->stage + static_cast<int64_t>(half) * pool->stage_slots * pool->slice_bytes,
                            pool->slice_bytes, 0};
    const hck::LaunchEvents ev = pool->prof_events();
    e = hck::launch_page_copy(src, dst, pool->slice_bytes, 1, false, pool->plan_dev,
                              static_cast<int32_t>(pool->plan.size()), nullptr, pool->copy_blocks, cs, ev);
    pool->prof_done(KV_KERNEL_PREFETCH_COPY, ev, e);
    if (e != hipSuccess) return hip_fail(e, "prefetch launch");
    e = hipEventRecord(pool->half_ready[half], cs);
    if (e == hipSuccess) e = hipEventRecord(pool->prefetch_done, cs);
    if (e != hipSuccess) return hip_fail(e, "hipEventRecord(prefetch)");
    pool->half_ready_pending[half] = true;
    pool->prefetch_pending = true;
    pool->half_layer[half] = layer;
    return KV_OK;
}

int paged_decode_gather_table(kv_pool* pool, const int32_t* sids, int32_t n, int32_t* table,
                              kv_stream_t stream) {
    if (!pool) return fail(KV_ERR_INVALID, "NULL pool");
    if (pool->meta) return fail(KV_ERR_INVALID, "metadata-only pool");
    if (n < 0 || n > kMaxDecodeBatch || (n > 0 && (!sids || !table)))
        return fail(KV_ERR_INVALID, "bad arguments");
    if (n == 0) return KV_OK;
    DeviceGuard g(pool->d.device);
    hipError_t e = hck::launch_gather_rows(pool->pt, pool->d.max_pages_per_session, pool->d.max_sessions,
                                           sids, n, table, pool->strm(stream));
    if (e != hipSuccess) return hip_fail(e, "gather launch");
    return KV_OK;
}

int paged_decode_partition(kv_pool* pool, const int32_t* seq_lens, int32_t batch, int32_t waves,
                           int32_t* slots_out, kv_stream_t stream) {
    if (!pool) return fail(KV_ERR_INVALID, "NULL pool");
    if (pool->meta) return fail(KV_ERR_INVALID, "metadata-only pool");
    if (batch < 0 || batch > kMaxDecodeBatch || waves < 1 || !slots_out || (batch > 0 && !seq_lens))
        return fail(KV_ERR_INVALID, "bad arguments");
    DeviceGuard g(pool->d.device);
    hipError_t e = hck::launch_partition(seq_lens, batch, pool->d.num_kv_heads, waves,
                                         hck::decode_group_waves(pool->d.num_kv_heads, waves),
                                         pool->d.max_pages_per_session, slots_out,
                                         pool->strm(stream));
    if (e != hipSuccess) return hip_fail(e, "partition launch");
    return KV_OK;
}

const char* kv_strerror(int status) {
    switch (status) {
        case KV_OK: return "ok";
        case KV_ERR_INVALID: return "invalid argument";
        case KV_ERR_STATE: return "session in the wrong state";
        case KV_ERR_NO_HOT_PAGES: return "hot pool exhausted";
        case KV_ERR_NO_COLD_PAGES: return "cold pool exhausted";
        case KV_ERR_HIP: return "HIP runtime error";
        case KV_ERR_OOM: return "out of memory";
        default: return "unknown status";
    }
}

const char* kv_last_error(void) { return g_err.c_str(); }

int kv_read_probe(const void* buf, size_t bytes, uint32_t* out, int32_t blocks, kv_stream_t stream) {
    if (!buf || !out || bytes == 0 || bytes % 16 || (reinterpret_cast<uintptr_t>(buf) & 15) || blocks < 1 ||
        blocks > (1 << 20))
        return fail(KV_ERR_INVALID, "bad arguments");
    hipError_t e = hck::launch_read_probe(buf, static_cast<int64_t>(bytes), out, blocks,
                                          static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "read probe launch");
    return KV_OK;
}

int kv_device_cu_slots(int32_t device, int32_t* xcds, int32_t* slots) {
    if (!xcds || !slots) return fail(KV_ERR_INVALID, "NULL output");
    int n = 0;
    hipError_t e = hipGetDeviceCount(&n);
    if (e != hipSuccess) return hip_fail(e, "device count");
    if (device < 0 || device >= n) return fail(KV_ERR_INVALID, "no such device");
    int cus = 0, x = 0;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&x, hipDeviceAttributeNumberOfXccs, device);
    if (e != hipSuccess) return hip_fail(e, "device attributes");
    if (x < 1 || cus < x || cus % x != 0) return fail(KV_ERR_INVALID, "CUs do not divide evenly over the XCDs");
    *xcds = x;
    *slots = cus / x;
    return KV_OK;
}

int kv_stream_create_cu_slots(int32_t device, int32_t slot_begin, int32_t slot_end, kv_stream_t* stream_out) {
    if (!stream_out) return fail(KV_ERR_INVALID, "NULL output");
    int32_t xcds = 0, slots = 0;
    const int rc = kv_device_cu_slots(device, &xcds, &slots);
    if (rc != KV_OK) return rc;
    if (slot_begin < 0 || slot_end > slots || slot_begin >= slot_end)
        return fail(KV_ERR_INVALID, "slot range outside [0, CUs per XCD)");
    // slot j of XCD x is mask bit x + xcds * j
    std::vector<uint32_t> mask((static_cast<size_t>(xcds) * slots + 31) / 32, 0u);
    for (int32_t j = slot_begin; j < slot_end; ++j)
        for (int32_t x = 0; x < xcds; ++x) {
            const int64_t bit = x + static_cast<int64_t>(xcds) * j;
            mask[bit / 32] |= 1u << (bit % 32);
        }
    DeviceGuard g(device);
    hipStream_t s = nullptr;
    const hipError_t e = hipExtStreamCreateWithCUMask(&s, static_cast<uint32_t>(mask.size()), mask.data());
    if (e != hipSuccess) return hip_fail(e, "CU-masked stream");
    *stream_out = s;
    return KV_OK;
}

int kv_stream_destroy(kv_stream_t stream) {
    if (!stream) return fail(KV_ERR_INVALID, "NULL stream");
    const hipError_t e = hipStreamDestroy(static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "stream destroy");
    return KV_OK;
}

int kv_pool_set_profiling(kv_pool* pool, int enable) {
    if (!pool) return fail(KV_ERR_INVALID, "NULL pool");
    if (pool->meta && enable) return fail(KV_ERR_INVALID, "metadata-only pool launches nothing");
    pool->profiling = enable != 0;
    return KV_OK;
}

int kv_pool_profile_read(kv_pool* pool, int32_t kernel_id, int32_t* launches, double* total_ms) {
    if (!pool || kernel_id < 0 || kernel_id >= KV_KERNEL_COUNT) return fail(KV_ERR_INVALID, "bad arguments");
    DeviceGuard g(pool->d.device);
    double sum = 0.0;
    int32_t count = 0;
    int rc = KV_OK;
    for (auto& r : pool->prof[kernel_id]) {
        float ms = 0.f;
        hipError_t e = hipEventSynchronize(r.stop);
        if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.start, r.stop);
        if (e != hipSuccess && rc == KV_OK) rc = hip_fail(e, "profiling event");
        sum += ms;
        ++count;
        pool->spare_events.push_back(r.start);
        pool->spare_events.push_back(r.stop);
    }
    pool->prof[kernel_id].clear();
    if (launches) *launches = count;
    if (total_ms) *total_ms = sum;
    return rc;
}

}  // extern "C"
