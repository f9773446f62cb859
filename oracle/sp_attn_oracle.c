/*
 * CPU oracle for session-prefill (SP) attention.  TEST INFRASTRUCTURE ONLY:
 * tests, the smoke check and the bench's CPU baseline call it; the product
 * path never does.  It shares no code with the HIP library.
 *
 * What it computes (plain definition, fp64, written out without blocking,
 * fusion or online rescaling):
 *
 *   SP admission prefills a continuation whose prefix KV is already on the
 *   device, recomputing only the new tail (Sections 3.4 and 4.3 of the paper:
 *   the admitted continuations are prefilled together as one batch; the
 *   shared prefix is already in device pages and only the tokens after it
 *   are computed, their KV going to fresh device pages).
 *   Sequence b has P_b cached tokens and S_b new tokens.  New token i sits
 *   at absolute position P_b + i and attends to keys 0 .. P_b + i
 *   (bottom-right causal alignment).  Query head h reads KV head
 *   g = h / (Hq / Hkv).  With sigma the softmax scale:
 *       s_j  = sigma * <q, k_j>,            j = 0 .. P_b + i
 *       o    = sum_j softmax(s)_j * v_j
 *       lse  = ln sum_j exp(s_j)
 *   Logical position t of sequence b is stored in the page pool at page
 *   block_tables[b][t / page_size], slot t mod page_size (the paged device
 *   KV layout that HKVR restores into, Appendix C, layer-first view:
 *   one layer's pool, pages within the layer).  Within a page the K pool is
 *   [Hkv][page_size][d] and the V pool [Hkv][d][page_size]:
 *       K(t, g, e) = k_pool[((page * Hkv + g) * page_size + slot) * d + e]
 *       V(t, g, e) = v_pool[((page * Hkv + g) * d + e) * page_size + slot]
 *
 * Precision: inputs are bf16 bit patterns widened exactly to double; every
 * product, sum, exp and log is double.  Softmax is two-pass (max, then
 * exp/sum), the textbook stable form.
 *
 * All functions return 0 on success and a negative value on a malformed
 * argument (out-of-range page id, bad geometry).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static double bf16_to_double(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Pool slot (flat index page * page_size + slot) of logical token t of
 * sequence b, or -1 if the block table entry is out of range. */
static int64_t slot_of(const int32_t *block_tables, int64_t bt_stride, int64_t b, int64_t t,
                       int64_t page_size, int64_t num_pages)
{
    int64_t page = block_tables[b * bt_stride + t / page_size];
    if (page < 0 || page >= num_pages)
        return -1;
    return page * page_size + t % page_size;
}

/* Flat offsets of element (g, e) of pool slot (page, slot). */
static int64_t k_index(int64_t page, int64_t slot, int64_t g, int64_t e, int64_t Hkv,
                       int64_t page_size, int64_t d)
{
    return ((page * Hkv + g) * page_size + slot) * d + e;
}

static int64_t v_index(int64_t page, int64_t slot, int64_t g, int64_t e, int64_t Hkv,
                       int64_t page_size, int64_t d)
{
    return ((page * Hkv + g) * d + e) * page_size + slot;
}

/*
 * Append: copy the K and V rows of every new token into its pool slot.
 * The new tokens of sequence b are rows off_b .. off_b + S_b - 1 of k_new /
 * v_new ([T][Hkv][d]); token i goes to logical position P_b + i.  Every
 * other pool slot keeps its bits.
 */
int oracle_append_kv(int32_t num_seqs, const int32_t *prefix_lens, const int32_t *suffix_lens,
                     const int32_t *block_tables, int64_t bt_stride, int32_t page_size,
                     int64_t num_pages, int32_t Hkv, int32_t d,
                     const uint16_t *k_new, const uint16_t *v_new,
                     uint16_t *k_pool, uint16_t *v_pool)
{
    int64_t off = 0;
    for (int32_t b = 0; b < num_seqs; ++b) {
        for (int64_t i = 0; i < suffix_lens[b]; ++i) {
            int64_t t = (int64_t)prefix_lens[b] + i;
            if (t / page_size >= bt_stride)
                return -1;
            int64_t flat = slot_of(block_tables, bt_stride, b, t, page_size, num_pages);
            if (flat < 0)
                return -1;
            int64_t page = flat / page_size, slot = flat % page_size;
            for (int64_t g = 0; g < Hkv; ++g)
                for (int64_t e = 0; e < d; ++e) {
                    int64_t src = ((off + i) * Hkv + g) * d + e;
                    k_pool[k_index(page, slot, g, e, Hkv, page_size, d)] = k_new[src];
                    v_pool[v_index(page, slot, g, e, Hkv, page_size, d)] = v_new[src];
                }
        }
        off += suffix_lens[b];
    }
    return 0;
}

/*
 * Gather: copy every logical token 0 .. P_b + S_b - 1 of every sequence
 * from the pool into contiguous rows [sum(P+S)][Hkv][d] (sequence-major),
 * bit for bit.
 */
int oracle_gather_kv(int32_t num_seqs, const int32_t *prefix_lens, const int32_t *suffix_lens,
                     const int32_t *block_tables, int64_t bt_stride, int32_t page_size,
                     int64_t num_pages, int32_t Hkv, int32_t d,
                     const uint16_t *k_pool, const uint16_t *v_pool,
                     uint16_t *k_out, uint16_t *v_out)
{
    int64_t off = 0;
    for (int32_t b = 0; b < num_seqs; ++b) {
        int64_t n = (int64_t)prefix_lens[b] + suffix_lens[b];
        for (int64_t t = 0; t < n; ++t) {
            if (t / page_size >= bt_stride)
                return -1;
            int64_t flat = slot_of(block_tables, bt_stride, b, t, page_size, num_pages);
            if (flat < 0)
                return -1;
            int64_t page = flat / page_size, slot = flat % page_size;
            for (int64_t g = 0; g < Hkv; ++g)
                for (int64_t e = 0; e < d; ++e) {
                    int64_t dst = ((off + t) * Hkv + g) * d + e;
                    k_out[dst] = k_pool[k_index(page, slot, g, e, Hkv, page_size, d)];
                    v_out[dst] = v_pool[v_index(page, slot, g, e, Hkv, page_size, d)];
                }
        }
        off += n;
    }
    return 0;
}

/* One query row against n contiguous double keys/values: two-pass softmax. */
static void attend_row(const double *qrow, const double *K, const double *V, int64_t n, int d,
                       double sigma, double *scores, double *o, double *lse)
{
    double m = -INFINITY;
    for (int64_t j = 0; j < n; ++j) {
        double dot = 0.0;
        for (int e = 0; e < d; ++e)
            dot += qrow[e] * K[j * d + e];
        scores[j] = sigma * dot;
        if (scores[j] > m)
            m = scores[j];
    }
    double l = 0.0;
    for (int e = 0; e < d; ++e)
        o[e] = 0.0;
    for (int64_t j = 0; j < n; ++j) {
        double w = exp(scores[j] - m);
        l += w;
        for (int e = 0; e < d; ++e)
            o[e] += w * V[j * d + e];
    }
    for (int e = 0; e < d; ++e)
        o[e] /= l;
    *lse = m + log(l);
}

/*
 * Shared driver: for each sequence b and KV head g, fetch K and V of
 * positions 0 .. P_b + S_b - 1 into contiguous double arrays through the
 * caller's fetch rule, then attend every requested query row of that group.
 *
 * rows == NULL means every row r = token * Hq + h in order; otherwise rows
 * lists num_rows flat row ids and output k belongs to rows[k].
 */
typedef int (*fetch_fn)(const void *ctx, int32_t b, int64_t t, int32_t g, uint16_t *krow,
                        uint16_t *vrow);

static int attention_driver(int32_t num_seqs, const int32_t *prefix_lens,
                            const int32_t *suffix_lens, int32_t Hq, int32_t Hkv, int32_t d,
                            double sigma, const uint16_t *q, fetch_fn fetch, const void *ctx,
                            int64_t num_rows, const int64_t *rows, double *o, double *lse)
{
    if (num_seqs < 0 || Hq <= 0 || Hkv <= 0 || d <= 0 || Hq % Hkv != 0)
        return -2;
    int32_t G = Hq / Hkv;
    int64_t T = 0;
    for (int32_t b = 0; b < num_seqs; ++b)
        T += suffix_lens[b];
    int64_t total_rows = rows ? num_rows : T * Hq;

    /* Token offset of each sequence, and the sequence of each token. */
    int64_t *tok_off = (int64_t *)malloc(sizeof(int64_t) * (size_t)(num_seqs + 1));
    if (!tok_off)
        return -3;
    tok_off[0] = 0;
    for (int32_t b = 0; b < num_seqs; ++b)
        tok_off[b + 1] = tok_off[b] + suffix_lens[b];

    int status = 0;
    for (int32_t b = 0; b < num_seqs && status == 0; ++b) {
        int64_t n = (int64_t)prefix_lens[b] + suffix_lens[b];
        if (suffix_lens[b] == 0)
            continue;
        double *K = (double *)malloc(sizeof(double) * (size_t)(n * d));
        double *V = (double *)malloc(sizeof(double) * (size_t)(n * d));
        if (!K || !V) {
            free(K);
            free(V);
            status = -3;
            break;
        }
        uint16_t *kr = (uint16_t *)malloc(sizeof(uint16_t) * (size_t)d);
        uint16_t *vr = (uint16_t *)malloc(sizeof(uint16_t) * (size_t)d);
        for (int32_t g = 0; g < Hkv && status == 0 && kr && vr; ++g) {
            for (int64_t t = 0; t < n; ++t) {
                if (fetch(ctx, b, t, g, kr, vr) != 0) {
                    status = -1;
                    break;
                }
                for (int e = 0; e < d; ++e) {
                    K[t * d + e] = bf16_to_double(kr[e]);
                    V[t * d + e] = bf16_to_double(vr[e]);
                }
            }
            if (status != 0)
                break;
#pragma omp parallel
            {
                double *scores = (double *)malloc(sizeof(double) * (size_t)n);
                double *qrow = (double *)malloc(sizeof(double) * (size_t)d);
#pragma omp for schedule(dynamic, 4)
                for (int64_t k = 0; k < total_rows; ++k) {
                    int64_t r = rows ? rows[k] : k;
                    int64_t token = r / Hq;
                    int32_t h = (int32_t)(r % Hq);
                    if (token < tok_off[b] || token >= tok_off[b + 1] || h / G != g)
                        continue;
                    int64_t i = token - tok_off[b];
                    int64_t visible = (int64_t)prefix_lens[b] + i + 1;
                    for (int e = 0; e < d; ++e)
                        qrow[e] = bf16_to_double(q[r * d + e]);
                    attend_row(qrow, K, V, visible, d, sigma, scores, o + k * d, lse + k);
                }
                free(scores);
                free(qrow);
            }
        }
        if (!kr || !vr)
            status = -3;
        free(kr);
        free(vr);
        free(K);
        free(V);
    }
    free(tok_off);
    return status;
}

struct paged_ctx {
    const int32_t *block_tables;
    int64_t bt_stride;
    int64_t page_size;
    int64_t num_pages;
    int32_t Hkv;
    int32_t d;
    const uint16_t *k_pool;
    const uint16_t *v_pool;
};

static int fetch_paged(const void *vctx, int32_t b, int64_t t, int32_t g, uint16_t *krow,
                       uint16_t *vrow)
{
    const struct paged_ctx *c = (const struct paged_ctx *)vctx;
    if (t / c->page_size >= c->bt_stride)
        return -1;
    int64_t flat = slot_of(c->block_tables, c->bt_stride, b, t, c->page_size, c->num_pages);
    if (flat < 0)
        return -1;
    int64_t page = flat / c->page_size, slot = flat % c->page_size;
    for (int64_t e = 0; e < c->d; ++e) {
        krow[e] = c->k_pool[k_index(page, slot, g, e, c->Hkv, c->page_size, c->d)];
        vrow[e] = c->v_pool[v_index(page, slot, g, e, c->Hkv, c->page_size, c->d)];
    }
    return 0;
}

/*
 * SP attention reading K/V through block tables from the pools (layouts
 * in the header comment; the pool must already hold
 * the new tokens' K/V, i.e. append has run).  q is [T][Hq][d]; o is
 * [rows][d] and lse [rows] (natural log).  sm_scale <= 0 selects 1/sqrt(d).
 */
int oracle_sp_attention(int32_t num_seqs, const int32_t *prefix_lens, const int32_t *suffix_lens,
                        const int32_t *block_tables, int64_t bt_stride, int32_t page_size,
                        int64_t num_pages, int32_t Hq, int32_t Hkv, int32_t d, double sm_scale,
                        const uint16_t *q, const uint16_t *k_pool, const uint16_t *v_pool,
                        int64_t num_rows, const int64_t *rows, double *o, double *lse)
{
    struct paged_ctx c = {block_tables, bt_stride, page_size, num_pages, Hkv, d, k_pool, v_pool};
    double sigma = sm_scale > 0.0 ? sm_scale : 1.0 / sqrt((double)d);
    if (page_size <= 0)
        return -2;
    return attention_driver(num_seqs, prefix_lens, suffix_lens, Hq, Hkv, d, sigma, q,
                            fetch_paged, &c, num_rows, rows, o, lse);
}

struct contig_ctx {
    const int64_t *kv_off;
    int32_t Hkv;
    int32_t d;
    const uint16_t *k_all;
    const uint16_t *v_all;
};

static int fetch_contig(const void *vctx, int32_t b, int64_t t, int32_t g, uint16_t *krow,
                        uint16_t *vrow)
{
    const struct contig_ctx *c = (const struct contig_ctx *)vctx;
    int64_t base = ((c->kv_off[b] + t) * c->Hkv + g) * (int64_t)c->d;
    memcpy(krow, c->k_all + base, sizeof(uint16_t) * (size_t)c->d);
    memcpy(vrow, c->v_all + base, sizeof(uint16_t) * (size_t)c->d);
    return 0;
}

/*
 * The same attention, reading K/V of sequence b from contiguous rows
 * k_all/v_all [sum_b (P_b + S_b)][Hkv][d] (sequence-major, positions in
 * order).  Independent of any page layout.
 */
int oracle_attention_contiguous(int32_t num_seqs, const int32_t *prefix_lens,
                                const int32_t *suffix_lens, int32_t Hq, int32_t Hkv, int32_t d,
                                double sm_scale, const uint16_t *q, const uint16_t *k_all,
                                const uint16_t *v_all, int64_t num_rows, const int64_t *rows,
                                double *o, double *lse)
{
    int64_t *kv_off = (int64_t *)malloc(sizeof(int64_t) * (size_t)(num_seqs + 1));
    if (!kv_off)
        return -3;
    kv_off[0] = 0;
    for (int32_t b = 0; b < num_seqs; ++b)
        kv_off[b + 1] = kv_off[b] + prefix_lens[b] + suffix_lens[b];
    struct contig_ctx c = {kv_off, Hkv, d, k_all, v_all};
    double sigma = sm_scale > 0.0 ? sm_scale : 1.0 / sqrt((double)d);
    int rc = attention_driver(num_seqs, prefix_lens, suffix_lens, Hq, Hkv, d, sigma, q,
                              fetch_contig, &c, num_rows, rows, o, lse);
    free(kv_off);
    return rc;
}
