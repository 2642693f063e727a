/*
 * Oracle (test infrastructure only): plain fp64 paged grouped-query decode
 * attention.  Only the tests, the smoke check and the benchmark's CPU baseline
 * may call it; the GPU library never links or calls it, and it shares no code
 * with that library.
 *
 * What it computes is the textbook definition the paper relies on: decoding
 * attends to the cached keys and values of all past tokens (Sec. II, first
 * paragraph), which are kept in fixed-size blocks of a paged cache (Sec. II,
 * same paragraph, after vLLM's PagedAttention).  For session b with L tokens,
 * query head h and its KV head g = h / (Hq / Hkv):
 *
 *   s_t   = scale * sum_i q[b][h][i] * k_t[i]               t = 0 .. L-1
 *   m     = max_t s_t
 *   w_t   = exp(s_t - m),   Z = sum_t w_t
 *   out   = sum_t (w_t / Z) * v_t
 *
 * where token t lives in page page_table[b][t / P], slot t % P.  L = 0 gives a
 * zero output.  Everything is evaluated in double precision; bf16 and float32
 * inputs are widened exactly.
 *
 * Pool layout (documented by the library header; re-derived here on its own):
 * a page is [layer][kv_head][K tile, V tile]; a tile holds P tokens x D dims.
 *   K tile element (t, d): index ((d / x) * P + t) * x + (d % x), x = 16 / elt
 *   V tile element (t, d): index d * P + t
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORACLE_BF16 = 0, ORACLE_F32 = 1 };

typedef struct {
    int num_layers;
    int num_kv_heads;
    int head_dim;
    int page_size;
    int dtype;
} oracle_layout;

static int elt_bytes(int dtype) { return dtype == ORACLE_BF16 ? 2 : 4; }

static double widen(const uint8_t* p, int dtype) {
    if (dtype == ORACLE_BF16) {
        uint16_t h;
        memcpy(&h, p, 2);
        uint32_t bits = (uint32_t)h << 16;
        float f;
        memcpy(&f, &bits, 4);
        return (double)f;
    }
    float f;
    memcpy(&f, p, 4);
    return (double)f;
}

long oracle_page_bytes(const oracle_layout* L) {
    return (long)L->num_layers * L->num_kv_heads * 2 * L->page_size * L->head_dim * elt_bytes(L->dtype);
}

/* Byte offset of one K (kind 0) or V (kind 1) element inside the pool. */
long oracle_elem_offset(const oracle_layout* L, long page, int layer, int head, int kind, int t, int d) {
    const int e = elt_bytes(L->dtype);
    const long tile = (long)L->page_size * L->head_dim * e;
    long off = page * oracle_page_bytes(L) + ((long)(layer * L->num_kv_heads + head) * 2 + kind) * tile;
    long idx;
    if (kind == 0) {
        const int x = 16 / e;
        idx = ((long)(d / x) * L->page_size + t) * x + (d % x);
    } else {
        idx = (long)d * L->page_size + t;
    }
    return off + idx * e;
}

/*
 * Returns 0 on success, -1 on a bad argument, -2 if a page id used by a valid
 * token is outside [0, num_pages).
 * out: [batch][num_q_heads][head_dim] doubles.
 * weights (nullable): [batch][num_q_heads][weights_stride] doubles, w_t / Z.
 */
int oracle_paged_attention(const void* pool, long num_pages, const oracle_layout* L, int layer,
                           int batch, int num_q_heads, const void* q, const int32_t* page_table,
                           long pt_stride, const int32_t* seq_lens, double scale, double* out,
                           double* weights, long weights_stride, int num_threads) {
    if (!pool || !L || !q || !page_table || !seq_lens || !out) return -1;
    if (L->num_kv_heads <= 0 || num_q_heads % L->num_kv_heads != 0) return -1;
    if (layer < 0 || layer >= L->num_layers) return -1;
    const int D = L->head_dim, P = L->page_size, e = elt_bytes(L->dtype);
    const int G = num_q_heads / L->num_kv_heads;
    const uint8_t* base = (const uint8_t*)pool;
    const uint8_t* qb = (const uint8_t*)q;
    int status = 0;
#ifdef _OPENMP
    if (num_threads > 0) omp_set_num_threads(num_threads);
#else
    (void)num_threads;
#endif
#pragma omp parallel for schedule(dynamic, 1)
    for (long row = 0; row < (long)batch * num_q_heads; ++row) {
        const int b = (int)(row / num_q_heads), h = (int)(row % num_q_heads);
        const int g = h / G;
        const int Lb = seq_lens[b];
        double* o = out + row * D;
        for (int i = 0; i < D; ++i) o[i] = 0.0;
        if (Lb <= 0 || (long)(Lb + P - 1) / P > pt_stride) {
            if (Lb < 0 || (long)(Lb + P - 1) / P > pt_stride) {
#pragma omp atomic write
                status = -1;
            }
            continue;
        }
        double* s = (double*)malloc(sizeof(double) * (size_t)Lb);
        double* qd = (double*)malloc(sizeof(double) * (size_t)D);
        for (int i = 0; i < D; ++i) qd[i] = widen(qb + ((long)row * D + i) * e, L->dtype);
        int bad = 0;
        for (int t = 0; t < Lb && !bad; ++t) {
            const long page = page_table[(long)b * pt_stride + t / P];
            if (page < 0 || page >= num_pages) { bad = 1; break; }
            double acc = 0.0;
            for (int i = 0; i < D; ++i)
                acc += qd[i] * widen(base + oracle_elem_offset(L, page, layer, g, 0, t % P, i), L->dtype);
            s[t] = scale * acc;
        }
        if (bad) {
#pragma omp atomic write
            status = -2;
            free(s);
            free(qd);
            continue;
        }
        double m = s[0];
        for (int t = 1; t < Lb; ++t) if (s[t] > m) m = s[t];
        double Z = 0.0;
        for (int t = 0; t < Lb; ++t) { s[t] = exp(s[t] - m); Z += s[t]; }
        for (int t = 0; t < Lb; ++t) {
            const long page = page_table[(long)b * pt_stride + t / P];
            const double w = s[t] / Z;
            if (weights) weights[row * weights_stride + t] = w;
            for (int i = 0; i < D; ++i)
                o[i] += w * widen(base + oracle_elem_offset(L, page, layer, g, 1, t % P, i), L->dtype);
        }
        free(s);
        free(qd);
    }
    return status;
}

/*
 * Write one session's logical K and V of one layer ([seq_len][num_kv_heads]
 * [head_dim], elements of the pool's dtype) into a host pool: token t goes to
 * page pages[t / P], slot t % P, at the offsets oracle_elem_offset gives.  The
 * same job as the numpy packer (oracle.pack_pool), for sizes numpy is slow on.
 */
int oracle_pack_session(void* pool, const oracle_layout* L, int layer, const int32_t* pages, long seq_len,
                        const void* k, const void* v) {
    if (!pool || !L || (seq_len > 0 && (!pages || !k || !v))) return -1;
    const int e = elt_bytes(L->dtype), H = L->num_kv_heads, D = L->head_dim, P = L->page_size;
    uint8_t* base = (uint8_t*)pool;
    const uint8_t* kb = (const uint8_t*)k;
    const uint8_t* vb = (const uint8_t*)v;
#pragma omp parallel for schedule(static)
    for (long t = 0; t < seq_len; ++t) {
        const long page = pages[t / P];
        for (int g = 0; g < H; ++g)
            for (int d = 0; d < D; ++d) {
                const long src = ((t * H + g) * (long)D + d) * e;
                memcpy(base + oracle_elem_offset(L, page, layer, g, 0, (int)(t % P), d), kb + src, (size_t)e);
                memcpy(base + oracle_elem_offset(L, page, layer, g, 1, (int)(t % P), d), vb + src, (size_t)e);
            }
    }
    return 0;
}
