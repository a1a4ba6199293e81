/*
 * TEST INFRASTRUCTURE ONLY -- the CPU oracle for batched tree verification.
 *
 * A plain, slow, obviously correct evaluation of what the verification step
 * of SLO-customised speculative decoding computes (section 4.3, step 4: the
 * target model scores every node of every request's draft token tree in one
 * pass, then the accepted path decides the committed tokens).  Only the test
 * suite, the smoke check and the benchmark's CPU-baseline leg may load it;
 * the product path never does.  It shares no code, header or table with the
 * HIP library.
 *
 * Arithmetic: every floating-point input (bf16 bit patterns or float32) is
 * widened exactly to double and all sums, maxima and exponentials are taken
 * in double.  Parallelism: OpenMP over independent (node, head) pairs or
 * requests only; each result is computed by one thread in a fixed order, so
 * results do not depend on the thread count.
 *
 * Definitions followed (the paper gives no verification listing; these are
 * the definitions it states):
 *  - draft token tree (section 2): nodes are tokens, the root is the last
 *    generated token, every root-to-node path is a candidate continuation;
 *  - path probability f(v) (section 3, Theorem 1): acceptance is decided per
 *    root-to-v path, so a node sees exactly its own root-to-node path;
 *  - verification (section 4.3 step 4; section 5.1): the target model
 *    produces logits for every node, and the verified tokens are read off
 *    those logits;
 *  - parents precede children in a tree (Appendix B), so local parent ids
 *    satisfy 0 <= parent[i] < i with the root at local id 0.
 *
 * Readings where the paper is silent (greedy argmax acceptance, ties,
 * accept-length convention, GQA head mapping) are stated at each function.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ---------------------------------------------------------------- helpers */

static double widen_bf16(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static double value_at(const void *base, int64_t idx, int is_bf16)
{
    if (is_bf16)
        return widen_bf16(((const uint16_t *)base)[idx]);
    return (double)((const float *)base)[idx];
}

/* A request's tree is well formed when it has a root at local id 0 whose
 * parent is -1 and every other node's parent is an earlier node. */
static int tree_well_formed(const int32_t *par, int32_t n)
{
    if (n < 1 || par[0] != -1)
        return 0;
    for (int32_t i = 1; i < n; ++i)
        if (par[i] < 0 || par[i] >= i)
            return 0;
    return 1;
}

/* Root-to-node path of local node i: path[0] = 0 (root), path[k] = i.
 * Returns k + 1, the number of nodes on the path (depth + 1). */
static int32_t root_path(const int32_t *par, int32_t i, int32_t *path)
{
    int32_t len = 0;
    for (int32_t v = i; v != -1; v = par[v])
        ++len;
    int32_t k = len;
    for (int32_t v = i; v != -1; v = par[v])
        path[--k] = v;
    return len;
}

static int32_t request_of(int32_t B, const int32_t *indptr, int32_t node)
{
    for (int32_t r = 0; r < B; ++r)
        if (node >= indptr[r] && node < indptr[r + 1])
            return r;
    return -1;
}

/* ------------------------------------------------------------- threads */

void oracle_set_num_threads(int32_t n)
{
#ifdef _OPENMP
    if (n > 0)
        omp_set_num_threads(n);
#else
    (void)n;
#endif
}

int32_t oracle_get_num_threads(void)
{
#ifdef _OPENMP
    return (int32_t)omp_get_max_threads();
#else
    return 1;
#endif
}

/* ----------------------------------------------------------- attention */

/*
 * Tree attention for the selected nodes (all q-heads of each).
 *
 * For node i of request r and q-head h (kv-head g = h / (Hq / Hkv), i.e.
 * contiguous head groups), the keys and values are, in this order:
 *   1. the request's cached prefix, positions t = 0 .. L_r - 1, read from
 *      page block_table[r][t / ps], slot t % ps, head g;
 *   2. the tree nodes on i's root-to-node path, root first, i last, read
 *      from k_tree / v_tree at head g.
 * Output: softmax over s_j = sm_scale * <q_i,h, k_j> applied to the v_j,
 * i.e. ordinary attention of one query over the sequence "prefix followed
 * by the node's root-to-node path" (section 2: a root-to-node path is a
 * candidate continuation; section 4.3 step 4: all nodes are scored in one
 * pass).
 *
 * Layouts: q [T, Hq, D]; k_tree, v_tree [T, Hkv, D];
 * k_pages, v_pages [num_pages, Hkv, ps, D]; block_table [B, bt_stride].
 * out [num_sel, Hq, D] in double.
 *
 * Returns 0, or -1 when a selected node is out of range, its request's tree
 * is malformed, or a needed block-table entry is outside [0, num_pages).
 */
int32_t oracle_tree_attn(int32_t B, const int32_t *indptr, const int32_t *parent,
                         const int32_t *prefix_len, const int32_t *block_table,
                         int64_t bt_stride, int32_t num_pages,
                         const void *q, const void *k_tree, const void *v_tree,
                         const void *k_pages, const void *v_pages, int32_t is_bf16,
                         int32_t Hq, int32_t Hkv, int32_t D, int32_t ps, double sm_scale,
                         int32_t num_sel, const int32_t *sel, double *out)
{
    if (Hq <= 0 || Hkv <= 0 || Hq % Hkv != 0 || D <= 0 || ps <= 0)
        return -1;
    const int32_t G = Hq / Hkv;
    /* Validate everything first; the parallel loop then cannot fail. */
    for (int32_t s = 0; s < num_sel; ++s) {
        int32_t r = request_of(B, indptr, sel[s]);
        if (r < 0)
            return -1;
        if (!tree_well_formed(parent + indptr[r], indptr[r + 1] - indptr[r]))
            return -1;
        int32_t L = prefix_len[r];
        if (L < 0)
            return -1;
        for (int32_t t = 0; t < L; t += ps) {
            int32_t page = block_table[(int64_t)r * bt_stride + t / ps];
            if (page < 0 || page >= num_pages)
                return -1;
        }
    }

    const int64_t tasks = (int64_t)num_sel * Hq;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t task = 0; task < tasks; ++task) {
        const int32_t s = (int32_t)(task / Hq), h = (int32_t)(task % Hq);
        const int32_t node = sel[s];
        const int32_t r = request_of(B, indptr, node);
        const int32_t base = indptr[r];
        const int32_t *par = parent + base;
        const int32_t L = prefix_len[r];
        const int32_t g = h / G;
        int32_t path[130];
        int32_t *pathbuf = (indptr[r + 1] - base) + 1 > 130
                               ? (int32_t *)malloc(sizeof(int32_t) * (size_t)(indptr[r + 1] - base + 1))
                               : path;
        const int32_t plen = root_path(par, node - base, pathbuf);
        const int64_t nkeys = (int64_t)L + plen;
        double *score = (double *)malloc(sizeof(double) * (size_t)(nkeys > 0 ? nkeys : 1));
        const int64_t qoff = ((int64_t)node * Hq + h) * D;

        /* scores over the prefix, then over the root-to-node path */
        for (int64_t t = 0; t < L; ++t) {
            const int32_t page = block_table[(int64_t)r * bt_stride + t / ps];
            const int64_t koff = (((int64_t)page * Hkv + g) * ps + t % ps) * D;
            double acc = 0.0;
            for (int32_t d = 0; d < D; ++d)
                acc += value_at(q, qoff + d, is_bf16) * value_at(k_pages, koff + d, is_bf16);
            score[t] = sm_scale * acc;
        }
        for (int32_t m = 0; m < plen; ++m) {
            const int64_t koff = ((int64_t)(base + pathbuf[m]) * Hkv + g) * D;
            double acc = 0.0;
            for (int32_t d = 0; d < D; ++d)
                acc += value_at(q, qoff + d, is_bf16) * value_at(k_tree, koff + d, is_bf16);
            score[L + m] = sm_scale * acc;
        }

        /* softmax and weighted sum of values */
        double mx = -INFINITY;
        for (int64_t j = 0; j < nkeys; ++j)
            if (score[j] > mx)
                mx = score[j];
        double denom = 0.0;
        for (int64_t j = 0; j < nkeys; ++j) {
            score[j] = exp(score[j] - mx);
            denom += score[j];
        }
        double *o = out + ((int64_t)s * Hq + h) * D;
        for (int32_t d = 0; d < D; ++d)
            o[d] = 0.0;
        for (int64_t t = 0; t < L; ++t) {
            const int32_t page = block_table[(int64_t)r * bt_stride + t / ps];
            const int64_t voff = (((int64_t)page * Hkv + g) * ps + t % ps) * D;
            for (int32_t d = 0; d < D; ++d)
                o[d] += score[t] * value_at(v_pages, voff + d, is_bf16);
        }
        for (int32_t m = 0; m < plen; ++m) {
            const int64_t voff = ((int64_t)(base + pathbuf[m]) * Hkv + g) * D;
            for (int32_t d = 0; d < D; ++d)
                o[d] += score[L + m] * value_at(v_tree, voff + d, is_bf16);
        }
        for (int32_t d = 0; d < D; ++d)
            o[d] /= denom;

        free(score);
        if (pathbuf != path)
            free(pathbuf);
    }
    return 0;
}

/* -------------------------------------------------------------- argmax */

/*
 * Per-node vocabulary argmax of the verification logits (section 5.1: the
 * logits of every tree node come back from verification and the verified
 * tokens are identified from them; greedy reading: the target's choice at a
 * node is its highest-scoring token).
 *
 * Row i is logits[i * row_stride + 0 .. vocab - 1].  The scan keeps the
 * first position holding the largest value: a later position replaces the
 * best only when strictly greater, so ties go to the lowest index and +0 and
 * -0 compare equal.  Writes -1 for every row when vocab < 1.
 */
void oracle_node_argmax(const void *logits, int64_t row_stride, int32_t rows, int32_t vocab,
                        int32_t is_bf16, int32_t *out)
{
#pragma omp parallel for schedule(static)
    for (int32_t i = 0; i < rows; ++i) {
        if (vocab < 1) {
            out[i] = -1;
            continue;
        }
        const int64_t off = (int64_t)i * row_stride;
        int32_t best = 0;
        double best_v = value_at(logits, off, is_bf16);
        for (int32_t v = 1; v < vocab; ++v) {
            const double x = value_at(logits, off + v, is_bf16);
            if (x > best_v) {
                best_v = x;
                best = v;
            }
        }
        out[i] = best;
    }
}

/* -------------------------------------------------------------- accept */

/*
 * Output convention shared by both acceptance evaluations below.
 *
 * Reading of the paper (sections 2 and 4.3): the root is the last generated
 * token and counts as one accepted token (n_acc starts at 1); a non-root
 * node j matches when its draft token equals the target's argmax at its
 * parent; j is accepted when every non-root node on its root-to-node path
 * matches.  Let d* be the largest depth of an accepted node and i* the
 * smallest local id among accepted nodes of that depth.  Then
 *   accept_len[r]          = d* + 1
 *   accept_nodes[r][k]     = k-th node of the root..i* path   (k = 0..d*)
 *   accept_tokens[r][k]    = draft token of path node k + 1   (k < d*)
 *   accept_tokens[r][d*]   = argmax at i*  (the target's own next token)
 * and slots k > d* hold -1.  A request whose tree is malformed (no root at
 * local 0, or a parent not earlier than its child) or deeper than
 * max_accept - 1 gets accept_len -1 and all slots -1.
 */
static void clear_row(int32_t *row, int32_t n)
{
    for (int32_t k = 0; k < n; ++k)
        row[k] = -1;
}

static void emit(const int32_t *path, int32_t dstar, const int32_t *draft, const int32_t *amax,
                 int32_t base, int32_t *len, int32_t *tok, int32_t *nodes)
{
    *len = dstar + 1;
    for (int32_t k = 0; k <= dstar; ++k)
        nodes[k] = path[k];
    for (int32_t k = 0; k < dstar; ++k)
        tok[k] = draft[base + path[k + 1]];
    tok[dstar] = amax[base + path[dstar]];
}

/* Topological evaluation: one pass over the nodes in id order. */
void oracle_tree_accept(int32_t B, const int32_t *indptr, const int32_t *parent,
                        const int32_t *draft, const int32_t *amax, int32_t max_accept,
                        int32_t *accept_len, int32_t *accept_tokens, int32_t *accept_nodes)
{
#pragma omp parallel for schedule(dynamic, 16)
    for (int32_t r = 0; r < B; ++r) {
        const int32_t base = indptr[r], n = indptr[r + 1] - indptr[r];
        const int32_t *par = parent + base;
        int32_t *tok = accept_tokens + (int64_t)r * max_accept;
        int32_t *nodes = accept_nodes + (int64_t)r * max_accept;
        clear_row(tok, max_accept);
        clear_row(nodes, max_accept);
        accept_len[r] = -1;
        if (!tree_well_formed(par, n))
            continue;
        int32_t *depth = (int32_t *)malloc(sizeof(int32_t) * (size_t)n);
        unsigned char *acc = (unsigned char *)malloc((size_t)n);
        depth[0] = 0;
        acc[0] = 1;
        int32_t deepest = 0;
        for (int32_t i = 1; i < n; ++i) {
            const int32_t p = par[i];
            depth[i] = depth[p] + 1;
            acc[i] = (unsigned char)(acc[p] && draft[base + i] == amax[base + p]);
            if (depth[i] > deepest)
                deepest = depth[i];
        }
        if (deepest < max_accept) {
            int32_t best = 0;
            for (int32_t i = 1; i < n; ++i)
                if (acc[i] && depth[i] > depth[best])
                    best = i;
            int32_t *path = (int32_t *)malloc(sizeof(int32_t) * (size_t)(depth[best] + 1));
            root_path(par, best, path);
            emit(path, depth[best], draft, amax, base, &accept_len[r], tok, nodes);
            free(path);
        }
        free(depth);
        free(acc);
    }
}

/*
 * Brute-force evaluation: enumerate every root-to-leaf path, find on each
 * the longest prefix whose tokens all match (the target's argmax at each
 * node predicts the next node's draft token), and keep the longest prefix
 * over all leaves, ties broken by the smaller id of the prefix's last node.
 * Independent of oracle_tree_accept; the two are cross-checked in tests.
 */
void oracle_tree_accept_bruteforce(int32_t B, const int32_t *indptr, const int32_t *parent,
                                   const int32_t *draft, const int32_t *amax, int32_t max_accept,
                                   int32_t *accept_len, int32_t *accept_tokens,
                                   int32_t *accept_nodes)
{
#pragma omp parallel for schedule(dynamic, 16)
    for (int32_t r = 0; r < B; ++r) {
        const int32_t base = indptr[r], n = indptr[r + 1] - indptr[r];
        const int32_t *par = parent + base;
        int32_t *tok = accept_tokens + (int64_t)r * max_accept;
        int32_t *nodes = accept_nodes + (int64_t)r * max_accept;
        clear_row(tok, max_accept);
        clear_row(nodes, max_accept);
        accept_len[r] = -1;
        if (!tree_well_formed(par, n))
            continue;
        unsigned char *has_child = (unsigned char *)calloc((size_t)n, 1);
        for (int32_t i = 1; i < n; ++i)
            has_child[par[i]] = 1;
        int32_t *path = (int32_t *)malloc(sizeof(int32_t) * (size_t)n);
        int32_t *best_path = (int32_t *)malloc(sizeof(int32_t) * (size_t)n);
        int32_t best_m = -1, best_node = -1, longest = 0;
        for (int32_t leaf = 0; leaf < n; ++leaf) {
            if (has_child[leaf])
                continue;
            const int32_t len = root_path(par, leaf, path);
            if (len - 1 > longest)
                longest = len - 1;
            int32_t m = 0;
            while (m + 1 < len && draft[base + path[m + 1]] == amax[base + path[m]])
                ++m;
            if (m > best_m || (m == best_m && path[m] < best_node)) {
                best_m = m;
                best_node = path[m];
                memcpy(best_path, path, sizeof(int32_t) * (size_t)(m + 1));
            }
        }
        if (longest < max_accept)
            emit(best_path, best_m, draft, amax, base, &accept_len[r], tok, nodes);
        free(has_child);
        free(path);
        free(best_path);
    }
}
