/*
 * CPU oracle for the target-model tree-verification step.
 *
 * TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg may load this library. It shares no code,
 * header, table or helper with the GPU library; the two never include or
 * call each other.
 *
 * What it computes, and where the paper states it:
 *   - tree attention (§2.1: the draft tree is verified in one target pass
 *     under a tree-shaped attention mask; §8 cites SpecInfer's tree masking;
 *     §1: each decode step attends over every cached key): every node of a
 *     draft tree attends to the whole committed prefix of its sequence plus
 *     the tree nodes on its own root path (itself and its ancestors);
 *   - per-node greedy argmax over the vocabulary (§7.1: temperature 0);
 *   - greedy acceptance (§5.3: verification accepts one path of the draft
 *     tree and yields a bonus token; Alg. 2 calls it the ground-truth token):
 *     a node is accepted when its parent is accepted and its token equals the
 *     target's argmax at the parent; the deepest accepted node ends the path;
 *   - compaction of the accepted path's K/V rows into the paged cache
 *     (§1: the KV cache keeps the keys/values of committed tokens; rejected
 *     branches are discarded).
 *
 * Arithmetic is fp64 on exactly widened bf16 / fp32 inputs. Every function is
 * a direct transcription of the plain definition: loops, no blocking, no
 * fusion, no reordering beyond the definition. OpenMP only distributes
 * independent (sequence, node, head) items, so results do not depend on the
 * thread count.
 *
 * Readings of points the paper leaves open (each is also listed with the
 * design notes of this repository):
 *   - a node with parent -1 is a root: an already-trusted anchor that is
 *     always accepted (several roots form a forest);
 *   - a node sees itself (the visibility set is reflexive);
 *   - all prefix keys are visible to every node;
 *   - softmax scale defaults to 1/sqrt(D) when the caller passes scale <= 0;
 *   - query head h reads KV head floor(h / (Hq / Hkv));
 *   - argmax ties go to the lowest index, -0 equals +0, and the first NaN
 *     wins (as numpy.argmax does);
 *   - among accepted nodes the path ends at the deepest one, ties to the
 *     lowest node index;
 *   - accept_len counts path nodes including the root.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static double widen_bf16(uint16_t bits)
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

/* Threads the OpenMP loops below use from now on (results do not depend on it). */
void oracle_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n > 0)
        omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* Node count of sequence b: num_nodes[b] when given, else N. */
static int nodes_of(const int32_t *num_nodes, int N, int b)
{
    return num_nodes ? num_nodes[b] : N;
}

/* Argument checks shared by the attention entry points. Nodes at or past a
 * sequence's node count are padding: their parents are not looked at. */
static int attention_args_ok(const int32_t *page_table, const int32_t *kv_len,
                             const int32_t *parent, const int32_t *num_nodes, int B, int N,
                             int Hq, int Hkv, int D, int P, int max_pages, int num_pages)
{
    if (B < 0 || N < 1 || Hq < 1 || Hkv < 1 || D < 1 || P < 1 || Hq % Hkv != 0)
        return 0;
    for (int b = 0; b < B; ++b) {
        const int nb = nodes_of(num_nodes, N, b);
        if (nb < 0 || nb > N)
            return 0;
        int L = kv_len[b];
        if (L < 0 || (L + P - 1) / P > max_pages)
            return 0;
        for (int t = 0; t < L; t += P) {
            int pg = page_table[(long)b * max_pages + t / P];
            if (pg < 0 || pg >= num_pages)
                return 0;
        }
        for (int i = 0; i < nb; ++i) {
            int p = parent[(long)b * N + i];
            if (p < -1 || p >= i)
                return 0;
        }
    }
    return 1;
}

/* One output row of a padding node: zeros, and the log-sum-exp of an empty
 * key set. */
static void padding_row(int D, double *o, double *lse_out)
{
    for (int d = 0; d < D; ++d)
        o[d] = 0.0;
    if (lse_out)
        *lse_out = -INFINITY;
}

/* One output row: node i of sequence b, query head h. Writes D values to o
 * and the log-sum-exp to *lse_out (if not NULL). Returns 0, or -1 when its
 * scratch memory cannot be allocated (nothing written). */
static int attend_one(const uint16_t *q, const uint16_t *k_tree, const uint16_t *v_tree,
                       const uint16_t *k_cache, const uint16_t *v_cache,
                       const int32_t *page_table, const int32_t *kv_len, const int32_t *parent,
                       int N, int Hq, int Hkv, int D, int P, int max_pages, double scale, int b,
                       int i, int h, double *o, double *lse_out)
{
    const int G = Hq / Hkv;
    const int g = h / G;
    const int L = kv_len[b];
    const uint16_t *qrow = q + (((long)b * N + i) * Hq + h) * D;

    /* visible keys: the L prefix positions, then node i and its ancestors */
    int nvis = L;
    for (int j = i; j >= 0; j = parent[(long)b * N + j])
        ++nvis;
    const uint16_t **krow = malloc(sizeof(*krow) * (size_t)nvis);
    const uint16_t **vrow = malloc(sizeof(*vrow) * (size_t)nvis);
    double *s = malloc(sizeof(double) * (size_t)nvis);
    if (!krow || !vrow || !s) {
        free(krow);
        free(vrow);
        free(s);
        return -1;
    }

    int n = 0;
    for (int t = 0; t < L; ++t) {
        long pg = page_table[(long)b * max_pages + t / P];
        long off = ((pg * P + t % P) * Hkv + g) * D;
        krow[n] = k_cache + off;
        vrow[n] = v_cache + off;
        ++n;
    }
    for (int j = i; j >= 0; j = parent[(long)b * N + j]) {
        long off = (((long)b * N + j) * Hkv + g) * D;
        krow[n] = k_tree + off;
        vrow[n] = v_tree + off;
        ++n;
    }

    /* scores and their maximum */
    double m = -INFINITY;
    for (int j = 0; j < n; ++j) {
        double dot = 0.0;
        for (int d = 0; d < D; ++d)
            dot += widen_bf16(qrow[d]) * widen_bf16(krow[j][d]);
        s[j] = scale * dot;
        if (s[j] > m)
            m = s[j];
    }
    /* softmax-weighted sum of values */
    double denom = 0.0;
    for (int j = 0; j < n; ++j) {
        s[j] = exp(s[j] - m);
        denom += s[j];
    }
    /* o[d] = sum_j s_j v_j[d] / denom; each o[d] sums its terms in key order
     * j = 0, 1, ..., walking the value rows one after the other */
    for (int d = 0; d < D; ++d)
        o[d] = 0.0;
    for (int j = 0; j < n; ++j)
        for (int d = 0; d < D; ++d)
            o[d] += s[j] * widen_bf16(vrow[j][d]);
    for (int d = 0; d < D; ++d)
        o[d] /= denom;
    if (lse_out)
        *lse_out = m + log(denom);
    free(krow);
    free(vrow);
    free(s);
    return 0;
}

/* Tree-masked attention of every node's query heads over the paged prefix
 * plus the node's own root path. Outputs are fp64:
 *   out [B, N, Hq, D], lse [B, N, Hq] (natural log of sum_j exp(s_j)).
 * num_nodes (may be NULL: every sequence has N nodes) gives each sequence's
 * node count; rows of the nodes past it are padding (zeros, lse -inf) and no
 * padding input is read. Returns 0, or -1 on a malformed argument (nothing
 * written). */
int oracle_tree_attention(const uint16_t *q, const uint16_t *k_tree, const uint16_t *v_tree,
                          const uint16_t *k_cache, const uint16_t *v_cache,
                          const int32_t *page_table, const int32_t *kv_len,
                          const int32_t *parent, const int32_t *num_nodes, int B, int N, int Hq,
                          int Hkv, int D, int P, int max_pages, int num_pages, double scale,
                          double *out, double *lse)
{
    if (!attention_args_ok(page_table, kv_len, parent, num_nodes, B, N, Hq, Hkv, D, P, max_pages,
                           num_pages))
        return -1;
    if (!(scale > 0.0))
        scale = 1.0 / sqrt((double)D);

    int failed = 0;
#pragma omp parallel for collapse(3) schedule(dynamic, 4)
    for (int b = 0; b < B; ++b)
        for (int i = 0; i < N; ++i)
            for (int h = 0; h < Hq; ++h) {
                long row = ((long)b * N + i) * Hq + h;
                if (i >= nodes_of(num_nodes, N, b))
                    padding_row(D, out + row * D, lse ? lse + row : NULL);
                else if (attend_one(q, k_tree, v_tree, k_cache, v_cache, page_table, kv_len,
                                    parent, N, Hq, Hkv, D, P, max_pages, scale, b, i, h,
                                    out + row * D, lse ? lse + row : NULL) != 0) {
#pragma omp atomic write
                    failed = 1;
                }
            }
    return failed ? -2 : 0;
}

/* The same attention for a list of n_items (b, i, h) triples only (items is
 * [n_items][3]); row k of out_rows [n_items, D] and lse_rows [n_items]
 * belongs to item k. Used to check large workloads on sampled outputs. */
int oracle_tree_attention_rows(const uint16_t *q, const uint16_t *k_tree, const uint16_t *v_tree,
                               const uint16_t *k_cache, const uint16_t *v_cache,
                               const int32_t *page_table, const int32_t *kv_len,
                               const int32_t *parent, const int32_t *num_nodes, int B, int N,
                               int Hq, int Hkv, int D, int P, int max_pages, int num_pages,
                               double scale, const int32_t *items, int n_items, double *out_rows,
                               double *lse_rows)
{
    if (!attention_args_ok(page_table, kv_len, parent, num_nodes, B, N, Hq, Hkv, D, P, max_pages,
                           num_pages))
        return -1;
    for (int k = 0; k < n_items; ++k) {
        const int32_t *it = items + 3L * k;
        if (it[0] < 0 || it[0] >= B || it[1] < 0 || it[1] >= N || it[2] < 0 || it[2] >= Hq)
            return -1;
    }
    if (!(scale > 0.0))
        scale = 1.0 / sqrt((double)D);

    int failed = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int k = 0; k < n_items; ++k) {
        const int32_t *it = items + 3L * k;
        if (it[1] >= nodes_of(num_nodes, N, it[0]))
            padding_row(D, out_rows + (long)k * D, lse_rows ? lse_rows + k : NULL);
        else if (attend_one(q, k_tree, v_tree, k_cache, v_cache, page_table, kv_len, parent, N,
                            Hq, Hkv, D, P, max_pages, scale, it[0], it[1], it[2],
                            out_rows + (long)k * D, lse_rows ? lse_rows + k : NULL) != 0) {
#pragma omp atomic write
            failed = 1;
        }
    }
    return failed ? -2 : 0;
}

/* argmax over each of `rows` rows of V fp32 logits: the lowest index holding
 * the maximum under IEEE comparison (-0 == +0); the first NaN wins. */
void oracle_argmax(const float *logits, long rows, long V, int32_t *out)
{
#pragma omp parallel for schedule(static)
    for (long r = 0; r < rows; ++r) {
        const float *x = logits + r * V;
        long best = 0;
        if (!isnan(x[0])) {
            for (long v = 1; v < V; ++v) {
                if (isnan(x[v])) {
                    best = v;
                    break;
                }
                if (x[v] > x[best])
                    best = v;
            }
        }
        out[r] = (int32_t)best;
    }
}

/* Greedy longest accepted path and bonus token, per sequence.
 *   accepted(i) = parent(i) == -1, or accepted(parent(i)) and
 *                 draft(i) == argmax(parent(i));
 *   the path ends at the accepted node of greatest depth (lowest index on a
 *   tie) and runs root first; bonus = argmax at its last node.
 * num_nodes (may be NULL: N nodes each) limits each sequence to its first
 * nodes; a sequence with none accepts nothing (length 0, bonus -1).
 * Returns 0, or -1 on a malformed tree. */
int oracle_accept(const int32_t *draft, const int32_t *parent, const int32_t *amax,
                  const int32_t *num_nodes, int B, int N, int32_t *accept_len,
                  int32_t *accept_idx, int32_t *bonus)
{
    int status = 0;
    for (int b = 0; b < B; ++b) {
        const int32_t *par = parent + (long)b * N;
        const int32_t *tok = draft + (long)b * N;
        const int32_t *am = amax + (long)b * N;
        int nb = nodes_of(num_nodes, N, b);
        if (nb < 0 || nb > N) {
            status = -1;
            nb = 0;
        }
        int *acc = malloc(sizeof(int) * (size_t)N);
        int *depth = malloc(sizeof(int) * (size_t)N);
        if (!acc || !depth) {
            free(acc);
            free(depth);
            return -2;
        }
        int sel = -1;
        for (int i = 0; i < nb; ++i) {
            int p = par[i];
            if (p < -1 || p >= i) {
                status = -1;
                acc[i] = 0;
                depth[i] = 0;
                continue;
            }
            if (p < 0) {
                acc[i] = 1;
                depth[i] = 0;
            } else {
                acc[i] = acc[p] && tok[i] == am[p];
                depth[i] = depth[p] + 1;
            }
            if (acc[i] && (sel < 0 || depth[i] > depth[sel]))
                sel = i;
        }
        int len = sel < 0 ? 0 : depth[sel] + 1;
        accept_len[b] = len;
        for (int j = 0; j < N; ++j)
            accept_idx[(long)b * N + j] = -1;
        for (int j = sel, d = len - 1; d >= 0; j = par[j], --d)
            accept_idx[(long)b * N + d] = j;
        bonus[b] = sel < 0 ? -1 : am[sel];
        free(acc);
        free(depth);
    }
    return status;
}

/* Copy the accepted path's tree K/V rows into cache positions
 * kv_len[b] .. kv_len[b] + accept_len[b] - 1 through the page table.
 * Every other cache byte is left as it was. Returns 0, or -1 (nothing more
 * written for that row) when a destination page is outside the pool. */
int oracle_kv_compact(const uint16_t *k_tree, const uint16_t *v_tree, uint16_t *k_cache,
                      uint16_t *v_cache, const int32_t *page_table, const int32_t *kv_len,
                      const int32_t *accept_idx, const int32_t *accept_len, int B, int N,
                      int Hkv, int D, int P, int max_pages, int num_pages)
{
    int status = 0;
    const size_t row_bytes = sizeof(uint16_t) * (size_t)Hkv * (size_t)D;
    for (int b = 0; b < B; ++b)
        for (int j = 0; j < accept_len[b]; ++j) {
            int node = accept_idx[(long)b * N + j];
            int pos = kv_len[b] + j;
            int slot_page = pos / P;
            if (node < 0 || node >= N || slot_page >= max_pages) {
                status = -1;
                continue;
            }
            long pg = page_table[(long)b * max_pages + slot_page];
            if (pg < 0 || pg >= num_pages) {
                status = -1;
                continue;
            }
            long dst = (pg * P + pos % P) * Hkv * D;
            long src = ((long)b * N + node) * Hkv * D;
            memcpy(k_cache + dst, k_tree + src, row_bytes);
            memcpy(v_cache + dst, v_tree + src, row_bytes);
        }
    return status;
}
