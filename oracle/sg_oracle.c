/*
 * Plain CPU oracle of the selective KV-transfer hot path (SmartGen,
 * arXiv 2607.28150).  TEST INFRASTRUCTURE ONLY: the tests, the smoke check and
 * the bench's CPU-baseline leg load it; the product library never does, and
 * this file shares no code, header or table with it.
 *
 * Everything is written as the plain definition, in double precision, with
 * plain loops (no blocking, no fusion).  Floating-point inputs arrive as
 * float32 arrays: bf16 values widen to float32 exactly, so the oracle sees the
 * same numbers the GPU does.  Parallelism is OpenMP over independent units
 * (request, layer, KV head); each unit writes a disjoint part of the output.
 *
 * Conventions shared with the product interface (restated independently):
 *   unit (l, h, b): layer l, KV head h, request b; q head g reads KV head g / G.
 *   cu_seqlens[B+1]: token offsets of the requests inside T = sum N_b.
 *   cu_k[B+1]: offsets of the requests' selected rows inside K_total.
 *   K, V: [Lkv][Hkv][T][d]; the layer stride is passed explicitly in rows of d
 *   elements (Hkv*T for a per-layer source, 0 for one source shared by every
 *   layer).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

#define SGO_OK 0
#define SGO_EINVAL (-1)

int sgo_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void sgo_set_threads(int n) {
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* ------------------------------------------------------------------------ */
/* Importance score (Section 4.1, "selection frequency" importance; the
 * attention definition of Section 2.1).
 *
 * For unit (l, h, b) with prompt length N and window W, every q head g of the
 * group {h*G .. h*G+G-1} and every window row w (absolute position
 * p = N - W + w) contributes its causal softmax attention probability:
 *     z_j   = (1/sqrt(d)) * sum_c q[g][w][c] * K[h][j][c],   j <= p
 *     score_j += exp(z_j - max z) / sum_i exp(z_i - max z).
 * The row sums to one, so the unit's scores add up to G * W.
 */
int sgo_score(int B, int L, int Hq, int Hkv, int d, int W,
              const int32_t *cu_seqlens, int64_t T,
              const float *q_win, const float *k, int64_t k_layer_rows,
              double *scores)
{
    if (B <= 0 || L <= 0 || Hkv <= 0 || Hq % Hkv != 0 || d <= 0 || W <= 0) return SGO_EINVAL;
    const int G = Hq / Hkv;
    const double scale = 1.0 / sqrt((double)d);
    for (int b = 0; b < B; ++b)
        if (cu_seqlens[b + 1] - cu_seqlens[b] < W) return SGO_EINVAL;
    const int nunits = L * Hkv * B;
#pragma omp parallel for schedule(dynamic, 1)
    for (int u = 0; u < nunits; ++u) {
        const int b = u % B;
        const int h = (u / B) % Hkv;
        const int l = u / (B * Hkv);
        const int64_t N = cu_seqlens[b + 1] - cu_seqlens[b];
        const float *K = k + ((int64_t)l * k_layer_rows + (int64_t)h * T + cu_seqlens[b]) * d;
        double *S = scores + ((int64_t)l * Hkv + h) * T + cu_seqlens[b];
        double *z = (double *)malloc(sizeof(double) * (size_t)N);
        for (int64_t j = 0; j < N; ++j) S[j] = 0.0;
        for (int g = h * G; g < (h + 1) * G; ++g) {
            for (int w = 0; w < W; ++w) {
                const float *q = q_win + ((((int64_t)b * L + l) * Hq + g) * W + w) * d;
                const int64_t p = N - W + w;          /* absolute position of the row */
                double m = -INFINITY;
                for (int64_t j = 0; j <= p; ++j) {
                    double acc = 0.0;
                    for (int c = 0; c < d; ++c) acc += (double)q[c] * (double)K[j * d + c];
                    z[j] = acc * scale;
                    if (z[j] > m) m = z[j];
                }
                double sum = 0.0;
                for (int64_t j = 0; j <= p; ++j) sum += exp(z[j] - m);
                for (int64_t j = 0; j <= p; ++j) S[j] += exp(z[j] - m) / sum;
            }
        }
        free(z);
    }
    return SGO_OK;
}

/* ------------------------------------------------------------------------ */
/* Budgeted top-k (Section 2.3: each head of each request selects its own
 * top-k entries, giving a KV index of BH x k).
 *
 * Order: a larger score ranks first; equal scores rank by lower token index;
 * -0 equals +0 (plain value comparison); NaN ranks below every number.  The
 * first k of that order are emitted sorted by ascending token index.
 */
typedef struct { float s; int32_t i; } sgo_entry;

static int sgo_rank_cmp(const void *pa, const void *pb) {
    const sgo_entry *a = (const sgo_entry *)pa, *b = (const sgo_entry *)pb;
    const int an = isnan(a->s), bn = isnan(b->s);
    if (an != bn) return an ? 1 : -1;          /* NaN last */
    if (!an) {
        if (a->s > b->s) return -1;
        if (a->s < b->s) return 1;
    }
    return (a->i < b->i) ? -1 : (a->i > b->i);  /* ties: lower index first */
}

static int sgo_int_cmp(const void *pa, const void *pb) {
    const int32_t a = *(const int32_t *)pa, b = *(const int32_t *)pb;
    return (a < b) ? -1 : (a > b);
}

int sgo_topk(int B, int L, int Hkv, const int32_t *cu_seqlens, int64_t T,
             const int32_t *cu_k, int64_t K_total, const float *scores, int32_t *idx)
{
    for (int b = 0; b < B; ++b) {
        const int64_t N = cu_seqlens[b + 1] - cu_seqlens[b];
        const int64_t kk = cu_k[b + 1] - cu_k[b];
        if (kk < 0 || kk > N) return SGO_EINVAL;
    }
    if (cu_k[B] != K_total || cu_seqlens[B] != T) return SGO_EINVAL;
    const int nunits = L * Hkv * B;
#pragma omp parallel for schedule(dynamic, 1)
    for (int u = 0; u < nunits; ++u) {
        const int b = u % B;
        const int lh = u / B;
        const int64_t N = cu_seqlens[b + 1] - cu_seqlens[b];
        const int64_t kk = cu_k[b + 1] - cu_k[b];
        const float *s = scores + (int64_t)lh * T + cu_seqlens[b];
        int32_t *out = idx + (int64_t)lh * K_total + cu_k[b];
        sgo_entry *e = (sgo_entry *)malloc(sizeof(sgo_entry) * (size_t)(N > 0 ? N : 1));
        for (int64_t j = 0; j < N; ++j) { e[j].s = s[j]; e[j].i = (int32_t)j; }
        qsort(e, (size_t)N, sizeof(sgo_entry), sgo_rank_cmp);
        for (int64_t j = 0; j < kk; ++j) out[j] = e[j].i;
        qsort(out, (size_t)kk, sizeof(int32_t), sgo_int_cmp);
        free(e);
    }
    return SGO_OK;
}

/* ------------------------------------------------------------------------ */
/* Pack the selected rows into one transfer buffer (proactive transfer,
 * Section 4.1; a "row" of selected entries is BH x k x d, Section 4.2).
 *
 * Layout: [K rows | V rows | int32 index table].  Slot s of unit (l, h),
 * request b, i-th selected entry is s = (l*Hkv + h)*K_total + cu_k[b] + i; its
 * K row is K[l][h][cu_seqlens[b] + idx[s]].  An index outside [0, N_b)
 * produces an all-zero row.
 */
int sgo_pack(int B, int L, int Hkv, int d, int esize,
             const int32_t *cu_seqlens, int64_t T, const int32_t *cu_k, int64_t K_total,
             const void *k, const void *v, int64_t kv_layer_rows,
             const int32_t *idx, void *dst)
{
    if (esize != 2 && esize != 4) return SGO_EINVAL;
    const int64_t rowb = (int64_t)d * esize;
    const int64_t S = (int64_t)L * Hkv * K_total;
    unsigned char *Kd = (unsigned char *)dst;
    unsigned char *Vd = Kd + S * rowb;
    int32_t *Id = (int32_t *)(Vd + S * rowb);
    const unsigned char *Ks = (const unsigned char *)k;
    const unsigned char *Vs = (const unsigned char *)v;
    for (int l = 0; l < L; ++l)
        for (int h = 0; h < Hkv; ++h)
            for (int b = 0; b < B; ++b) {
                const int64_t N = cu_seqlens[b + 1] - cu_seqlens[b];
                for (int64_t i = 0; i < cu_k[b + 1] - cu_k[b]; ++i) {
                    const int64_t s = ((int64_t)l * Hkv + h) * K_total + cu_k[b] + i;
                    const int32_t t = idx[s];
                    Id[s] = t;
                    if (t < 0 || t >= N) {
                        memset(Kd + s * rowb, 0, (size_t)rowb);
                        memset(Vd + s * rowb, 0, (size_t)rowb);
                        continue;
                    }
                    const int64_t src = (int64_t)l * kv_layer_rows + (int64_t)h * T + cu_seqlens[b] + t;
                    memcpy(Kd + s * rowb, Ks + src * rowb, (size_t)rowb);
                    memcpy(Vd + s * rowb, Vs + src * rowb, (size_t)rowb);
                }
            }
    return SGO_OK;
}

/* ------------------------------------------------------------------------ */
/* KV index splitting and reordering (Algorithm 1, Section 4.2).
 *
 * Row r holds kv_index[row_off[r] .. row_off[r+1]); its mask row starts at
 * mask[mask_off[r]] and has mask_len[r] entries (0 pad, 1 local, 2 remote).
 *   (1) m_i <- mask[kv_index_i]  (an index outside the mask row, or a value
 *       other than 1 or 2, counts as 0);
 *   (4)(5) optional reordering: sort the row by m descending, stably, and
 *       permute kv_index the same way (remote entries first);
 *   (2) local  <- kv_index[m == 1];   (3) remote <- kv_index[m == 2].
 * Outputs share the input segmentation; unused tail slots are set to -1.
 */
typedef struct { int m; int64_t pos; } sgo_mpos;

static int sgo_mpos_desc(const void *pa, const void *pb) {
    const sgo_mpos *a = (const sgo_mpos *)pa, *b = (const sgo_mpos *)pb;
    if (a->m != b->m) return (a->m > b->m) ? -1 : 1;
    return (a->pos < b->pos) ? -1 : (a->pos > b->pos);   /* stable */
}

int sgo_split(int rows, const int32_t *row_off, const int32_t *kv_index,
              const int8_t *mask, const int64_t *mask_off, const int32_t *mask_len,
              int reorder, int32_t *out_index, int32_t *local, int32_t *remote,
              int32_t *n_local, int32_t *n_remote)
{
    if (reorder && !out_index) return SGO_EINVAL;
#pragma omp parallel for schedule(dynamic, 16)
    for (int r = 0; r < rows; ++r) {
        const int64_t o = row_off[r];
        const int64_t n = row_off[r + 1] - o;
        sgo_mpos *mp = (sgo_mpos *)malloc(sizeof(sgo_mpos) * (size_t)(n > 0 ? n : 1));
        int32_t *ix = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
        /* (1) gather the mask values of the required entries */
        for (int64_t i = 0; i < n; ++i) {
            const int32_t t = kv_index[o + i];
            int m = 0;
            if (t >= 0 && t < mask_len[r]) m = mask[mask_off[r] + t];
            if (m != 1 && m != 2) m = 0;
            mp[i].m = m;
            mp[i].pos = i;
            ix[i] = t;
        }
        if (reorder) {
            /* (4) sort each row of the mask descending; (5) apply the order */
            qsort(mp, (size_t)n, sizeof(sgo_mpos), sgo_mpos_desc);
            for (int64_t i = 0; i < n; ++i) ix[i] = kv_index[o + mp[i].pos];
            for (int64_t i = 0; i < n; ++i) out_index[o + i] = ix[i];
        }
        /* (2) local and (3) remote entries, in the (possibly reordered) row order */
        int64_t nl = 0, nr = 0;
        for (int64_t i = 0; i < n; ++i) {
            if (mp[i].m == 1) local[o + nl++] = ix[i];
            else if (mp[i].m == 2) remote[o + nr++] = ix[i];
        }
        for (int64_t i = nl; i < n; ++i) local[o + i] = -1;
        for (int64_t i = nr; i < n; ++i) remote[o + i] = -1;
        n_local[r] = (int32_t)nl;
        n_remote[r] = (int32_t)nr;
        free(mp);
        free(ix);
    }
    return SGO_OK;
}

/* ------------------------------------------------------------------------ */
/* On-demand fetch (parallel on-demand transfer, Section 4.2; the non-GDR
 * path of Section 4.4 receives remote rows in host memory first).
 *
 * Row r copies entries i < n_r (n_r = n_valid[r], or the whole segment when
 * n_valid is NULL) of its index segment.  Entry i names source row
 * src_row_base[r] + index[row_off[r] + i] (or + i when index is NULL) and goes
 * to logical row dst_start[r] + i of the row's paged destination:
 * pool row page_table[r*max_pages + l/P] + l%P.  Copies whose source, page or
 * pool row fall outside their arrays are skipped.
 */
int sgo_fetch(int rows, int esize, int d, const int32_t *row_off, const int32_t *index,
              const int32_t *n_valid, const int64_t *src_row_base, int64_t src_rows,
              const void *k_src, const void *v_src,
              const int32_t *page_table, int page_size, int max_pages, const int32_t *dst_start,
              void *k_pool, void *v_pool, int64_t pool_rows)
{
    if (page_size <= 0 || (esize != 2 && esize != 4)) return SGO_EINVAL;
    const int64_t rowb = (int64_t)d * esize;
    for (int r = 0; r < rows; ++r) {
        const int64_t seg = row_off[r + 1] - row_off[r];
        const int64_t n = n_valid ? n_valid[r] : seg;
        for (int64_t i = 0; i < n && i < seg; ++i) {
            const int64_t t = index ? index[row_off[r] + i] : i;
            const int64_t src = src_row_base[r] + t;
            const int64_t lrow = (int64_t)dst_start[r] + i;
            if (src < 0 || src >= src_rows || lrow < 0) continue;
            const int64_t p = lrow / page_size;
            if (p >= max_pages) continue;
            const int64_t dst = (int64_t)page_table[(int64_t)r * max_pages + p] + lrow % page_size;
            if (dst < 0 || dst >= pool_rows) continue;
            memcpy((unsigned char *)k_pool + dst * rowb, (const unsigned char *)k_src + src * rowb, (size_t)rowb);
            memcpy((unsigned char *)v_pool + dst * rowb, (const unsigned char *)v_src + src * rowb, (size_t)rowb);
        }
    }
    return SGO_OK;
}

/* ------------------------------------------------------------------------ */
/* Decode attention over a partial KV set (Section 2.1 attention; the order of
 * entries does not change the result, Section 4.2).
 *
 * For sequence b and q head g (KV head h = g / G) the set holds n = n_rows[b,h]
 * logical rows; logical row i lives at pool row page_table[b,h][i/P] + i%P.
 *     z_i = scale * q . k_i,   o = sum_i softmax(z)_i v_i.
 * No causal mask: a decode query sees every cached row.  Rows whose pool
 * index falls outside [0, pool_rows) are left out; an empty set gives o = 0.
 */
int sgo_decode_attn(int B, int Hq, int Hkv, int d, double scale, const float *q,
                    const float *k_pool, const float *v_pool, int64_t pool_rows,
                    const int32_t *page_table, const int32_t *n_rows, int page_size, int max_pages,
                    double *out)
{
    if (Hkv <= 0 || Hq % Hkv != 0 || page_size <= 0) return SGO_EINVAL;
    const int G = Hq / Hkv;
#pragma omp parallel for schedule(dynamic, 1)
    for (int bg = 0; bg < B * Hq; ++bg) {
        const int b = bg / Hq, g = bg % Hq, h = g / G;
        int64_t n = n_rows[(int64_t)b * Hkv + h];
        if (n > (int64_t)max_pages * page_size) n = (int64_t)max_pages * page_size;
        if (n < 0) n = 0;
        const int32_t *pt = page_table + ((int64_t)b * Hkv + h) * max_pages;
        const float *qv = q + ((int64_t)b * Hq + g) * d;
        double *o = out + ((int64_t)b * Hq + g) * d;
        double *z = (double *)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
        int64_t *row = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
        double m = -INFINITY;
        for (int64_t i = 0; i < n; ++i) {
            row[i] = (int64_t)pt[i / page_size] + i % page_size;
            if (row[i] < 0 || row[i] >= pool_rows) { row[i] = -1; continue; }
            double acc = 0.0;
            for (int c = 0; c < d; ++c) acc += (double)qv[c] * (double)k_pool[row[i] * d + c];
            z[i] = acc * scale;
            if (z[i] > m) m = z[i];
        }
        double sum = 0.0;
        for (int64_t i = 0; i < n; ++i)
            if (row[i] >= 0) sum += exp(z[i] - m);
        for (int c = 0; c < d; ++c) o[c] = 0.0;
        if (sum > 0.0) {
            for (int64_t i = 0; i < n; ++i) {
                if (row[i] < 0) continue;
                const double p = exp(z[i] - m) / sum;
                for (int c = 0; c < d; ++c) o[c] += p * (double)v_pool[row[i] * d + c];
            }
        }
        free(z);
        free(row);
    }
    return SGO_OK;
}

/* ------------------------------------------------------------------------ */
/* Block importance (Section 4.1, eq. 1), over measured per-entry scores.
 *
 * Request b with N tokens, layer l: the sequence is cut into M blocks of
 * Nb = ceil(N / M) tokens; block m holds tokens [m*Nb, min((m+1)*Nb, N)).
 * A block's entries E are its tokens in every KV head, and
 *     I[b][l][m] = +inf                                  for l = 0, 1
 *     I[b][l][m] = (1/|E|) * sum_{(h, t) in E} score[l][h][s0 + t]   otherwise.
 * A block with no tokens (trailing blocks when N is not a multiple of M)
 * has no mean; it gets -inf in layers >= 2 (never preferred).
 */
int sgo_block_importance(int B, int L, int Hkv, const int32_t *cu_seqlens, int64_t T, int M,
                         const float *scores, double *out)
{
    if (B < 1 || L < 1 || Hkv < 1 || M < 1 || T < 0) return SGO_EINVAL;
    if (cu_seqlens[0] != 0 || cu_seqlens[B] != T) return SGO_EINVAL;
    for (int b = 0; b < B; ++b) {
        const int64_t s0 = cu_seqlens[b], N = cu_seqlens[b + 1] - s0;
        if (N < 0) return SGO_EINVAL;
        const int64_t Nb = (N + M - 1) / M;
        for (int l = 0; l < L; ++l)
            for (int m = 0; m < M; ++m) {
                double *o = out + ((int64_t)b * L + l) * M + m;
                if (l < 2) { *o = INFINITY; continue; }
                const int64_t t0 = (int64_t)m * Nb;
                const int64_t t1 = t0 + Nb < N ? t0 + Nb : N;
                if (t1 <= t0) { *o = -INFINITY; continue; }
                double sum = 0.0;
                for (int h = 0; h < Hkv; ++h)
                    for (int64_t t = t0; t < t1; ++t)
                        sum += (double)scores[((int64_t)l * Hkv + h) * T + s0 + t];
                *o = sum / (double)((t1 - t0) * Hkv);
            }
    }
    return SGO_OK;
}

/* ------------------------------------------------------------------------ */
/* Block pack (proactive transfer of KV blocks, Section 4.1).
 *
 * One request (tokens [s0, s0 + N) of the source rows), blocks of
 * Nb = ceil(N / M) tokens.  Selected block s has flat id c = l*M + m.  Its
 * head-h rows go to slots (s*Hkv + h)*Nb + r, r < Nb, of the K region, from
 * K[l][h][s0 + m*Nb + r]; rows past the prompt end (and every row of an id
 * outside [0, L*M)) are zero.  Layout: [K rows | V rows | int32 ids].
 */
int sgo_pack_blocks(int L, int Hkv, int d, int esize, int64_t T, int64_t s0, int64_t N, int M,
                    const void *k, const void *v, int64_t kv_layer_rows, int nblk, const int32_t *ids,
                    void *dst)
{
    if (esize != 2 && esize != 4) return SGO_EINVAL;
    if (L < 1 || Hkv < 1 || M < 1 || N < 0 || nblk < 0) return SGO_EINVAL;
    const int64_t Nb = (N + M - 1) / M;
    const int64_t rowb = (int64_t)d * esize;
    const int64_t S = (int64_t)nblk * Hkv * Nb;
    unsigned char *Kd = (unsigned char *)dst;
    unsigned char *Vd = Kd + S * rowb;
    int32_t *Id = (int32_t *)(Vd + S * rowb);
    const unsigned char *Ks = (const unsigned char *)k;
    const unsigned char *Vs = (const unsigned char *)v;
    for (int s = 0; s < nblk; ++s) {
        const int32_t c = ids[s];
        Id[s] = c;
        const int ok = c >= 0 && (int64_t)c < (int64_t)L * M;
        const int l = ok ? c / M : 0, m = ok ? c % M : 0;
        for (int h = 0; h < Hkv; ++h)
            for (int64_t r = 0; r < Nb; ++r) {
                const int64_t slot = ((int64_t)s * Hkv + h) * Nb + r;
                const int64_t t = (int64_t)m * Nb + r;
                if (!ok || t >= N) {
                    memset(Kd + slot * rowb, 0, (size_t)rowb);
                    memset(Vd + slot * rowb, 0, (size_t)rowb);
                    continue;
                }
                const int64_t src = (int64_t)l * kv_layer_rows + (int64_t)h * T + s0 + t;
                memcpy(Kd + slot * rowb, Ks + src * rowb, (size_t)rowb);
                memcpy(Vd + slot * rowb, Vs + src * rowb, (size_t)rowb);
            }
    }
    return SGO_OK;
}

/* ------------------------------------------------------------------------ */
/* Speculative transfer (Section 4.3).  The prefill side pushes KV blocks that
 * the proactive transfer left behind into the decode side's KV store, in
 * importance order (eq. 1), and turns their KV mask entries local (Section
 * 4.2: mask 1 = local, 2 = remote).
 *
 * One request (tokens [s0, s0 + N) of T), blocks of Nb = ceil(N / M) tokens,
 * flat id c = l*M + m.  For each id of `ids` with 0 <= c < L*M, in order:
 *   for every KV head h and block token t = m*Nb + r < N:
 *     K_dst, V_dst row l*dst_layer_rows + h*T + s0 + t
 *         = K_src, V_src row l*src_layer_rows + h*T + s0 + t
 *     mask[(l*Hkv + h)*T + s0 + t] = 1
 *   rem[c] = NaN when rem is given: the block leaves the row of remaining
 *   importances, so a later top-k over that row ranks it last.
 * Other ids are skipped.
 */
int sgo_spec_push(int L, int Hkv, int d, int esize, int64_t T, int64_t s0, int64_t N, int M,
                  const void *k_src, const void *v_src, int64_t src_layer_rows,
                  void *k_dst, void *v_dst, int64_t dst_layer_rows,
                  int nblk, const int32_t *ids, int8_t *mask, float *rem)
{
    if (esize != 2 && esize != 4) return SGO_EINVAL;
    if (L < 1 || Hkv < 1 || M < 1 || N < 0 || nblk < 0 || s0 < 0 || s0 + N > T) return SGO_EINVAL;
    const int64_t Nb = (N + M - 1) / M;
    const int64_t rowb = (int64_t)d * esize;
    for (int s = 0; s < nblk; ++s) {
        const int32_t c = ids[s];
        if (c < 0 || (int64_t)c >= (int64_t)L * M) continue;
        const int l = c / M, m = c % M;
        for (int h = 0; h < Hkv; ++h)
            for (int64_t r = 0; r < Nb; ++r) {
                const int64_t t = (int64_t)m * Nb + r;
                if (t >= N) break;
                const int64_t src = (int64_t)l * src_layer_rows + (int64_t)h * T + s0 + t;
                const int64_t dst = (int64_t)l * dst_layer_rows + (int64_t)h * T + s0 + t;
                memcpy((unsigned char *)k_dst + dst * rowb, (const unsigned char *)k_src + src * rowb, (size_t)rowb);
                memcpy((unsigned char *)v_dst + dst * rowb, (const unsigned char *)v_src + src * rowb, (size_t)rowb);
                mask[((int64_t)l * Hkv + h) * T + s0 + t] = 1;
            }
        if (rem) rem[c] = NAN;
    }
    return SGO_OK;
}

/* ------------------------------------------------------------------------ */
/* On-demand fetch with reuse (Section 4.2; Section 5.3 compares against
 * reusing fetched entries).  The fetch of sgo_fetch, where each copied entry
 * is also kept in the decode side's KV store and its mask entry turns local,
 * so later steps load it on the local lane.
 *
 * Row r, entry i < n_r (as in sgo_fetch), t = index[row_off[r] + i]:
 *   src = src_row_base[r] + t; an entry with src outside [0, src_rows) is
 *   skipped entirely;
 *   pool: as sgo_fetch (logical row dst_start[r] + i through the page table),
 *   when page_table is given;
 *   keep: row keep_row_base[r] + t of k_keep / v_keep, when inside
 *   [0, keep_rows); only then, and when mask is given, 0 <= t < mask_len[r]
 *   and 0 <= mask_off[r] + t < mask_bytes: mask[mask_off[r] + t] = 1.
 */
int sgo_fetch_keep(int rows, int esize, int d, const int32_t *row_off, const int32_t *index,
                   const int32_t *n_valid, const int64_t *src_row_base, int64_t src_rows,
                   const void *k_src, const void *v_src,
                   const int32_t *page_table, int page_size, int max_pages, const int32_t *dst_start,
                   void *k_pool, void *v_pool, int64_t pool_rows,
                   const int64_t *keep_row_base, void *k_keep, void *v_keep, int64_t keep_rows,
                   int8_t *mask, int64_t mask_bytes, const int64_t *mask_off, const int32_t *mask_len)
{
    if ((esize != 2 && esize != 4) || !index) return SGO_EINVAL;
    if (page_table && page_size <= 0) return SGO_EINVAL;
    const int64_t rowb = (int64_t)d * esize;
    for (int r = 0; r < rows; ++r) {
        const int64_t seg = row_off[r + 1] - row_off[r];
        const int64_t n = n_valid ? n_valid[r] : seg;
        for (int64_t i = 0; i < n && i < seg; ++i) {
            const int64_t t = index[row_off[r] + i];
            const int64_t src = src_row_base[r] + t;
            if (src < 0 || src >= src_rows) continue;
            const unsigned char *ks = (const unsigned char *)k_src + src * rowb;
            const unsigned char *vs = (const unsigned char *)v_src + src * rowb;
            const int64_t lrow = (int64_t)dst_start[r] + i;
            if (page_table && lrow >= 0 && lrow / page_size < max_pages) {
                const int64_t dst = (int64_t)page_table[(int64_t)r * max_pages + lrow / page_size] + lrow % page_size;
                if (dst >= 0 && dst < pool_rows) {
                    memcpy((unsigned char *)k_pool + dst * rowb, ks, (size_t)rowb);
                    memcpy((unsigned char *)v_pool + dst * rowb, vs, (size_t)rowb);
                }
            }
            const int64_t kr = keep_row_base[r] + t;
            if (kr < 0 || kr >= keep_rows) continue;
            memcpy((unsigned char *)k_keep + kr * rowb, ks, (size_t)rowb);
            memcpy((unsigned char *)v_keep + kr * rowb, vs, (size_t)rowb);
            if (mask && t >= 0 && t < mask_len[r] && mask_off[r] + t >= 0 && mask_off[r] + t < mask_bytes)
                mask[mask_off[r] + t] = 1;
        }
    }
    return SGO_OK;
}

/* ------------------------------------------------------------------------ */
/* Selection-frequency score under a threshold selector (Section 4.1 defines a
 * KV entry's importance as how often the decode-time selector picks it; the
 * selector of the evaluation, InfiniGen with alpha = 5 (Section 5.1), picks
 * the keys whose attention logit is within alpha of the row's maximum).  The
 * window rows stand in for decode queries, as in sgo_score:
 *     z_j = (1/sqrt(d)) * q[g][w] . K[h][j]  for j <= p,   m = max_j z_j,
 *     count_j += [z_j >= m - alpha]
 * over the G q heads of the group and the W rows, an integer in [0, G*W].
 * When `near` is given, near_j counts the rows with |z_j - (m - alpha)| <= eps:
 * the decisions that rounding of z could flip.
 */
int sgo_score_count(int B, int L, int Hq, int Hkv, int d, int W,
                    const int32_t *cu_seqlens, int64_t T,
                    const float *q_win, const float *k, int64_t k_layer_rows,
                    double alpha, double eps, int32_t *counts, int32_t *near)
{
    if (B <= 0 || L <= 0 || Hkv <= 0 || Hq % Hkv != 0 || d <= 0 || W <= 0 || !(alpha >= 0.0)) return SGO_EINVAL;
    const int G = Hq / Hkv;
    const double scale = 1.0 / sqrt((double)d);
    for (int b = 0; b < B; ++b)
        if (cu_seqlens[b + 1] - cu_seqlens[b] < W) return SGO_EINVAL;
    const int nunits = L * Hkv * B;
#pragma omp parallel for schedule(dynamic, 1)
    for (int u = 0; u < nunits; ++u) {
        const int b = u % B;
        const int h = (u / B) % Hkv;
        const int l = u / (B * Hkv);
        const int64_t N = cu_seqlens[b + 1] - cu_seqlens[b];
        const float *K = k + ((int64_t)l * k_layer_rows + (int64_t)h * T + cu_seqlens[b]) * d;
        int32_t *C = counts + ((int64_t)l * Hkv + h) * T + cu_seqlens[b];
        int32_t *E = near ? near + ((int64_t)l * Hkv + h) * T + cu_seqlens[b] : NULL;
        double *z = (double *)malloc(sizeof(double) * (size_t)N);
        for (int64_t j = 0; j < N; ++j) {
            C[j] = 0;
            if (E) E[j] = 0;
        }
        for (int g = h * G; g < (h + 1) * G; ++g)
            for (int w = 0; w < W; ++w) {
                const float *q = q_win + ((((int64_t)b * L + l) * Hq + g) * W + w) * d;
                const int64_t p = N - W + w;
                double m = -INFINITY;
                for (int64_t j = 0; j <= p; ++j) {
                    double acc = 0.0;
                    for (int c = 0; c < d; ++c) acc += (double)q[c] * (double)K[j * d + c];
                    z[j] = acc * scale;
                    if (z[j] > m) m = z[j];
                }
                const double thr = m - alpha;
                for (int64_t j = 0; j <= p; ++j) {
                    if (z[j] >= thr) C[j] += 1;
                    if (E && fabs(z[j] - thr) <= eps) E[j] += 1;
                }
            }
        free(z);
    }
    return SGO_OK;
}

/* ------------------------------------------------------------------------ */
/* Selection-frequency score under a top-share selector (Section 4.1 defines a
 * KV entry's importance as how often the selector picks it; Section 5.1 sets a
 * maximum selection ratio of 20%).  Window row w of q head g sees the
 * n = p + 1 keys j <= p = N - W + w and picks its top share of them:
 *     k   = max(1, min(n, floor(n * ratio_bp / 10000)))
 *     thr = the k-th largest of z_0 .. z_p   (z as in sgo_score_count)
 *     count_j += [z_j >= thr]                (every key tied with thr is picked)
 * an integer in [0, G*W].  `near` counts the rows with |z_j - thr| <= eps.
 */
static int cmp_desc(const void *a, const void *b) {
    const double x = *(const double *)a, y = *(const double *)b;
    return (x < y) - (x > y);
}

int sgo_score_topshare(int B, int L, int Hq, int Hkv, int d, int W,
                       const int32_t *cu_seqlens, int64_t T,
                       const float *q_win, const float *k, int64_t k_layer_rows,
                       int ratio_bp, double eps, int32_t *counts, int32_t *near)
{
    if (B <= 0 || L <= 0 || Hkv <= 0 || Hq % Hkv != 0 || d <= 0 || W <= 0 || ratio_bp < 1 || ratio_bp > 10000)
        return SGO_EINVAL;
    const int G = Hq / Hkv;
    const double scale = 1.0 / sqrt((double)d);
    for (int b = 0; b < B; ++b)
        if (cu_seqlens[b + 1] - cu_seqlens[b] < W) return SGO_EINVAL;
    const int nunits = L * Hkv * B;
#pragma omp parallel for schedule(dynamic, 1)
    for (int u = 0; u < nunits; ++u) {
        const int b = u % B;
        const int h = (u / B) % Hkv;
        const int l = u / (B * Hkv);
        const int64_t N = cu_seqlens[b + 1] - cu_seqlens[b];
        const float *K = k + ((int64_t)l * k_layer_rows + (int64_t)h * T + cu_seqlens[b]) * d;
        int32_t *C = counts + ((int64_t)l * Hkv + h) * T + cu_seqlens[b];
        int32_t *E = near ? near + ((int64_t)l * Hkv + h) * T + cu_seqlens[b] : NULL;
        double *z = (double *)malloc(sizeof(double) * (size_t)N);
        double *sorted = (double *)malloc(sizeof(double) * (size_t)N);
        for (int64_t j = 0; j < N; ++j) {
            C[j] = 0;
            if (E) E[j] = 0;
        }
        for (int g = h * G; g < (h + 1) * G; ++g)
            for (int w = 0; w < W; ++w) {
                const float *q = q_win + ((((int64_t)b * L + l) * Hq + g) * W + w) * d;
                const int64_t p = N - W + w;
                const int64_t n = p + 1;
                for (int64_t j = 0; j <= p; ++j) {
                    double acc = 0.0;
                    for (int c = 0; c < d; ++c) acc += (double)q[c] * (double)K[j * d + c];
                    z[j] = acc * scale;
                    sorted[j] = z[j];
                }
                int64_t kk = n * (int64_t)ratio_bp / 10000;
                if (kk < 1) kk = 1;
                if (kk > n) kk = n;
                qsort(sorted, (size_t)n, sizeof(double), cmp_desc);
                const double thr = sorted[kk - 1];
                for (int64_t j = 0; j <= p; ++j) {
                    if (z[j] >= thr) C[j] += 1;
                    if (E && fabs(z[j] - thr) <= eps) E[j] += 1;
                }
            }
        free(sorted);
        free(z);
    }
    return SGO_OK;
}

/* ------------------------------------------------------------------------ */
/* Decode-time dynamic selection (Section 2.3: the selector picks each step's
 * KV entries from the decode query; Section 5.1: alpha = 5 and a maximum KV
 * selection ratio of 20%).  For request b, layer l and KV head h, with the G q
 * heads of its group and the request's N keys:
 *     z[g][j] = (1/sqrt(d)) * q[b][l][g] . K[h][j],   m_g = max_j z[g][j]
 *     r_j     = max_g (z[g][j] - m_g)          (<= 0, and 0 at each head's maximum)
 *     S       = { j : r_j >= -alpha }          (some head of the group picks j)
 * If |S| exceeds cap_b = cu_cap[b+1] - cu_cap[b], the cap_b entries of S with
 * the largest r_j are kept (ties: lower j).  The kept ids go ascending to
 * idx[l][h][cu_cap[b] ...], n_sel[(b*L + l)*Hkv + h] counts them, and the rest
 * of the segment is -1.  r_out ([L][Hkv][T], optional) receives r.
 * q: [B][L][Hq][d]; K: [Lkv][Hkv][T][d] with the given layer stride.  The
 * logit scale is an argument: 1/sqrt(d) for whole rows; for a partial set of
 * channels (InfiniGen speculates with 30% of them, Section 5.1) the rows hold
 * only those channels and the scale stays that of the full head.
 */
typedef struct { double r; int32_t j; } sgo_rj;

static int sgo_rj_cmp(const void *pa, const void *pb) {
    const sgo_rj *a = (const sgo_rj *)pa, *b = (const sgo_rj *)pb;
    if (a->r > b->r) return -1;
    if (a->r < b->r) return 1;
    return (a->j < b->j) ? -1 : (a->j > b->j);
}

static int sgo_i32_cmp(const void *pa, const void *pb) {
    const int32_t a = *(const int32_t *)pa, b = *(const int32_t *)pb;
    return (a > b) - (a < b);
}

int sgo_decode_select(int B, int L, int Hq, int Hkv, int d, const float *q,
                      const int32_t *cu_seqlens, int64_t T, const float *k, int64_t k_layer_rows,
                      const int32_t *cu_cap, int64_t K_cap, double alpha, double scale,
                      int32_t *idx, int32_t *n_sel, double *r_out)
{
    if (B <= 0 || L <= 0 || Hkv <= 0 || Hq % Hkv != 0 || d <= 0 || !(alpha >= 0.0) || !(scale > 0.0))
        return SGO_EINVAL;
    const int G = Hq / Hkv;
    const int nunits = L * Hkv * B;
#pragma omp parallel for schedule(dynamic, 1)
    for (int u = 0; u < nunits; ++u) {
        const int b = u % B;
        const int h = (u / B) % Hkv;
        const int l = u / (B * Hkv);
        const int64_t N = cu_seqlens[b + 1] - cu_seqlens[b];
        const int64_t cap = cu_cap[b + 1] - cu_cap[b];
        const float *K = k + ((int64_t)l * k_layer_rows + (int64_t)h * T + cu_seqlens[b]) * d;
        int32_t *out = idx + ((int64_t)l * Hkv + h) * K_cap + cu_cap[b];
        double *r = (double *)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1));
        double *z = (double *)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1));
        for (int64_t j = 0; j < N; ++j) r[j] = -INFINITY;
        for (int g = h * G; g < (h + 1) * G; ++g) {
            const float *qg = q + (((int64_t)b * L + l) * Hq + g) * d;
            double m = -INFINITY;
            for (int64_t j = 0; j < N; ++j) {
                double acc = 0.0;
                for (int c = 0; c < d; ++c) acc += (double)qg[c] * (double)K[j * d + c];
                z[j] = acc * scale;
                if (z[j] > m) m = z[j];
            }
            for (int64_t j = 0; j < N; ++j)
                if (z[j] - m > r[j]) r[j] = z[j] - m;
        }
        if (r_out)
            for (int64_t j = 0; j < N; ++j) r_out[((int64_t)l * Hkv + h) * T + cu_seqlens[b] + j] = r[j];
        sgo_rj *s = (sgo_rj *)malloc(sizeof(sgo_rj) * (size_t)(N > 0 ? N : 1));
        int64_t ns = 0;
        for (int64_t j = 0; j < N; ++j)
            if (r[j] >= -alpha) {
                s[ns].r = r[j];
                s[ns].j = (int32_t)j;
                ++ns;
            }
        if (ns > cap) {
            qsort(s, (size_t)ns, sizeof(sgo_rj), sgo_rj_cmp);
            ns = cap;
        }
        int32_t *ids = (int32_t *)malloc(sizeof(int32_t) * (size_t)(ns > 0 ? ns : 1));
        for (int64_t i = 0; i < ns; ++i) ids[i] = s[i].j;
        qsort(ids, (size_t)ns, sizeof(int32_t), sgo_i32_cmp);
        for (int64_t i = 0; i < cap; ++i) out[i] = i < ns ? ids[i] : -1;
        n_sel[((int64_t)b * L + l) * Hkv + h] = (int32_t)ns;
        free(ids);
        free(s);
        free(z);
        free(r);
    }
    return SGO_OK;
}
