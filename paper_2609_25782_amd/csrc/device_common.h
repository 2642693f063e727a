// Device-side helpers shared by the library's kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hck {

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));

constexpr int kPageTokens = 16;
constexpr int kWave = 64;
constexpr int kBlockThreads = 256;
constexpr int kBlockWaves = kBlockThreads / kWave;

// Pages a row of `seq_len` tokens occupies, clamped to the row stride; rows
// with a non-positive length occupy none.
__device__ __forceinline__ int row_pages(int32_t seq_len, int64_t stride) {
    if (seq_len <= 0) return 0;
    const int64_t n = (static_cast<int64_t>(seq_len) + kPageTokens - 1) / kPageTokens;
    return static_cast<int>(n < stride ? n : stride);
}

// s_pref[b] = sum of row_pages over rows < b, for b = 0 .. batch (exclusive
// prefix sum plus the total).  All kThreads threads of the block must call it;
// the caller synchronises before reading s_pref.
template <int kThreads = kBlockThreads>
__device__ inline void block_prefix_pages(const int32_t* __restrict__ seq_lens, int batch,
                                          int64_t stride, int32_t* s_pref) {
    __shared__ int32_t s_wave_sum[kThreads / kWave];
    const int tid = threadIdx.x;
    const int per = (batch + kThreads - 1) / kThreads;
    const int lo = min(batch, tid * per);
    const int hi = min(batch, lo + per);
    int sum = 0;
    for (int b = lo; b < hi; ++b) sum += row_pages(seq_lens[b], stride);
    int x = sum;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const int y = __shfl_up(x, o);
        if ((tid & (kWave - 1)) >= o) x += y;
    }
    if ((tid & (kWave - 1)) == kWave - 1) s_wave_sum[tid / kWave] = x;
    __syncthreads();
    int base = 0;
    for (int w = 0; w < tid / kWave; ++w) base += s_wave_sum[w];
    int run = base + x - sum;
    for (int b = lo; b < hi; ++b) {
        s_pref[b] = run;
        run += row_pages(seq_lens[b], stride);
    }
    if (tid == kThreads - 1) s_pref[batch] = run;
}

// One piece of the decode work split: worker `k` handles pages [p0, p1) of
// row b, head group g (of `heads` per row); its partial results go to slot
// k + b * heads + g (scaled by the waves of a worker, see the decode kernel).
struct Piece {
    int b, g, p0, p1, slot;
};

// Wave-uniform read of an LDS word (all lanes read the same address); keeps
// values derived from it in scalar registers.
__device__ __forceinline__ int32_t lds_uniform(const int32_t* p) {
    return __builtin_amdgcn_readfirstlane(*p);
}

// Units are (row, head group, page) triples ordered by row, then head group,
// then page; worker k of `workers` owns units
// [floor(k T / workers), floor((k + 1) T / workers)).
__device__ __forceinline__ void wave_units(int64_t total_units, int worker, int workers, int64_t& u0,
                                           int64_t& u1) {
    u0 = static_cast<int64_t>(worker) * total_units / workers;
    u1 = static_cast<int64_t>(worker + 1) * total_units / workers;
}

// LDS read used by piece_at: readfirstlane when every lane of the wave asks
// for the same unit (decode), a plain per-lane read otherwise (partition table).
template <bool kWaveUniform>
__device__ __forceinline__ int32_t lds_read(const int32_t* p) {
    if constexpr (kWaveUniform) return lds_uniform(p);
    return *p;
}

// The piece of worker `worker` that starts at unit u (< total), ending no later
// than u_end; rows have `heads` head groups.
template <bool kWaveUniform>
__device__ __forceinline__ Piece piece_at(const int32_t* s_pref, int batch, int heads,
                                          int worker, int64_t u, int64_t u_end) {
    // largest row b with heads * s_pref[b] <= u; it has at least one page
    const int64_t target = u / heads;
    int lo = 0, hi = batch - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (lds_read<kWaveUniform>(s_pref + mid) <= target) lo = mid; else hi = mid - 1;
    }
    Piece pc;
    pc.b = lo;
    const int32_t first = lds_read<kWaveUniform>(s_pref + lo);
    const int nb = lds_read<kWaveUniform>(s_pref + lo + 1) - first;
    const int64_t rel = u - static_cast<int64_t>(first) * heads;
    pc.g = static_cast<int>(rel / nb);
    pc.p0 = static_cast<int>(rel % nb);
    const int64_t seg_end = u + (nb - pc.p0);
    const int64_t e = seg_end < u_end ? seg_end : u_end;
    pc.p1 = pc.p0 + static_cast<int>(e - u);
    pc.slot = worker + lo * heads + pc.g;
    return pc;
}

}  // namespace hck
