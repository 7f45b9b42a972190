/*
 * CPU oracle for hyperbatch GNN data preparation (AGNES, arXiv 2601.01473).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU-baseline
 * leg of the benchmark load this code.  It shares no source with the GPU library:
 * its Philox, its sampling and its relabelling are written here independently.
 *
 * What is computed (paper Sec. 3.1 and Alg. 1; where the paper is silent, the
 * conventions listed further down):
 *   For every minibatch j of a hyperbatch (global index m = mb_base + j) and for
 *   every hop l = 0..L-1, every node already in the minibatch is a request;
 *   each request v draws min(deg(v), f_l) distinct neighbour positions uniformly
 *   without replacement (Sec. 3.1, "randomly samples only a subset"), the union
 *   of the minibatch's nodes and the sampled neighbours forms the next set
 *   (Alg. 1, N_out accumulated by union; Eq. (1) needs h_v itself, so a node
 *   stays in its own next set), and each hop is emitted as a CSR block whose
 *   column ids are local ids in the minibatch's node list.  Finally the feature
 *   rows of every node of every minibatch are gathered into one contiguous
 *   buffer (Sec. 3.4(2), Alg. 1 gathering loop).
 *
 * Conventions fixed here (the paper is silent on them):
 *   - RNG: Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC 2011), key (seed, 0),
 *     counter (i >> 2, v, m, l); word i of a request is output lane (i & 3).
 *   - Integer in [0, n): high 64 bits of the 128-bit product w * n
 *     (Lemire, "Fast random integer generation in an interval", 2019), no
 *     rejection step.
 *   - Subset: Floyd's algorithm (Bentley and Floyd, CACM 30(9), 1987).
 *   - A CSR row lists its neighbours in ascending edge position.
 *   - Local ids: targets in the given order, then each hop's new nodes in
 *     ascending global id.
 *
 * Two orders of work are provided: the plain per-minibatch, per-node loop
 * (oracle_minibatch) and the block-bucketed hyperbatch order of Alg. 1
 * (oracle_hyperbatch_blocked).  They must produce identical results.
 */
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef unsigned __int128 u128;

/* ------------------------------------------------------------------ Philox */

/* Philox4x64 constants (Salmon et al. 2011, Sec. 4: multipliers and the
 * golden-ratio / sqrt(3)-1 Weyl increments of the key schedule). */
#define PHILOX_M0 0xD2E7470EE14C6C93ULL
#define PHILOX_M1 0xCA5A826395121157ULL
#define PHILOX_W0 0x9E3779B97F4A7C15ULL
#define PHILOX_W1 0xBB67AE8584CAA73BULL

/* Philox4x64 with 10 rounds: out = Philox(ctr, key). */
void oracle_philox4x64_10(const uint64_t ctr_in[4], const uint64_t key_in[2], uint64_t out[4]) {
    uint64_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
    uint64_t k0 = key_in[0], k1 = key_in[1];
    for (int round = 0; round < 10; round++) {
        if (round > 0) { k0 += PHILOX_W0; k1 += PHILOX_W1; }
        u128 p0 = (u128)PHILOX_M0 * c0;
        u128 p1 = (u128)PHILOX_M1 * c2;
        uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0;
        uint64_t hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
        uint64_t n0 = hi1 ^ c1 ^ k0;
        uint64_t n1 = lo1;
        uint64_t n2 = hi0 ^ c3 ^ k1;
        uint64_t n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Integer in [0, n) from a 64-bit word: floor(w * n / 2^64). */
uint64_t oracle_uniform_below(uint64_t w, uint64_t n) {
    return (uint64_t)(((u128)w * (u128)n) >> 64);
}

/* Random word i of the request (node v, minibatch m, hop l) under `seed`. */
uint64_t oracle_draw_word(uint64_t seed, int64_t v, int64_t m, int64_t l, int64_t i) {
    uint64_t ctr[4] = {(uint64_t)i >> 2, (uint64_t)v, (uint64_t)m, (uint64_t)l};
    uint64_t key[2] = {seed, 0};
    uint64_t out[4];
    oracle_philox4x64_10(ctr, key, out);
    return out[i & 3];
}

/* ------------------------------------------------------------------ Floyd */

static int cmp_i64(const void* a, const void* b) {
    int64_t x = *(const int64_t*)a, y = *(const int64_t*)b;
    return (x > y) - (x < y);
}

/*
 * Floyd's subset algorithm, driven by explicit draws: for i = 0..k-1 let
 * t = n - k + i; draw d_i in [0, t]; insert t if d_i is already chosen, else
 * insert d_i.  Writes the k chosen positions in ascending order.  Returns k, or
 * -1 if a draw is out of its range.
 */
int64_t oracle_floyd_from_draws(int64_t n, int64_t k, const uint64_t* draws, int64_t* out) {
    for (int64_t i = 0; i < k; i++) {
        int64_t t = n - k + i;
        int64_t d = (int64_t)draws[i];
        if (draws[i] > (uint64_t)t) return -1;
        int present = 0;
        for (int64_t s = 0; s < i; s++)
            if (out[s] == d) { present = 1; break; }
        out[i] = present ? t : d;
    }
    qsort(out, (size_t)k, sizeof(int64_t), cmp_i64);
    return k;
}

/*
 * Positions sampled for node v (degree deg) at hop l of minibatch m with fanout f:
 * k = min(deg, f) positions in [0, deg), ascending.  Returns k.
 */
int64_t oracle_sample_positions(int64_t deg, int64_t f, uint64_t seed, int64_t v, int64_t m,
                                int64_t l, int64_t* out) {
    int64_t k = deg < f ? deg : f;
    uint64_t* draws = (uint64_t*)malloc((size_t)(k > 0 ? k : 1) * sizeof(uint64_t));
    for (int64_t i = 0; i < k; i++) {
        int64_t t = deg - k + i;
        draws[i] = oracle_uniform_below(oracle_draw_word(seed, v, m, l, i), (uint64_t)(t + 1));
    }
    oracle_floyd_from_draws(deg, k, draws, out);
    free(draws);
    return k;
}

/* ------------------------------------------------------------------ helpers */

static int cmp_i32(const void* a, const void* b) {
    int32_t x = *(const int32_t*)a, y = *(const int32_t*)b;
    return (x > y) - (x < y);
}

enum { ORACLE_OK = 0, ORACLE_INVALID = 1, ORACLE_CAPACITY = 2, ORACLE_NOMEM = 3 };

/*
 * Append to the node list the nodes of cg[0..n) that are not yet in it, in
 * ascending global id; id[] maps global id -> local id (-1 when absent).
 * *count is updated in place.  Returns 0, or -1 when cap_nodes would be exceeded.
 */
static int union_new_sorted(const int32_t* cg, int64_t n, int32_t* nodes, int64_t* count,
                            int64_t cap_nodes, int32_t* id) {
    int32_t* tmp = (int32_t*)malloc((size_t)(n > 0 ? n : 1) * sizeof(int32_t));
    if (!tmp) return -1;
    memcpy(tmp, cg, (size_t)n * sizeof(int32_t));
    qsort(tmp, (size_t)n, sizeof(int32_t), cmp_i32);
    for (int64_t i = 0; i < n; i++) {
        if (i > 0 && tmp[i] == tmp[i - 1]) continue;
        int32_t u = tmp[i];
        if (id[u] >= 0) continue;
        if (*count >= cap_nodes) { free(tmp); return -1; }
        id[u] = (int32_t)*count;
        nodes[(*count)++] = u;
    }
    free(tmp);
    return 0;
}

/*
 * One minibatch, plain order: every hop, every node of the minibatch in local-id
 * order, sampled on its own.
 *
 * Inputs: CSR (offsets[num_nodes+1] int64, indices), the B targets, fanouts[L],
 * seed, and the global minibatch index m.  id_scratch: num_nodes int32 entries,
 * all -1 on entry; restored to -1 on return.
 * Outputs: nodes[cap_nodes] (local-id order), layer_sizes[L+1]
 * (|D_0| = B, then the node count after each hop), edge_counts[L]; per hop l
 * the row_ptr (layer_sizes[l]+1 entries, from 0) and col / col_global
 * (edge_counts[l] entries) are appended to row_ptr / col / col_global in hop
 * order.  col_global may be NULL.
 */
int oracle_minibatch(int64_t num_nodes, const int64_t* offsets, const int32_t* indices,
                     const int32_t* targets, int32_t B, const int32_t* fanouts, int32_t L,
                     uint64_t seed, int64_t m, int64_t cap_nodes, int32_t* nodes,
                     int32_t* layer_sizes, int64_t* edge_counts, int64_t cap_rowptr,
                     int32_t* row_ptr, int64_t cap_edges, int32_t* col, int32_t* col_global,
                     int32_t* id_scratch) {
    int32_t* id = id_scratch;
    int64_t count = 0, rp_used = 0, e_used = 0;
    int rc = ORACLE_OK;
    int64_t* pos = NULL;

    /* D_0: the targets, in the given order (Alg. 1, minibatch assignment) */
    for (int32_t r = 0; r < B; r++) {
        int32_t v = targets[r];
        if (v < 0 || v >= num_nodes || id[v] >= 0) { rc = ORACLE_INVALID; goto done; }
        if (count >= cap_nodes) { rc = ORACLE_CAPACITY; goto done; }
        id[v] = (int32_t)count;
        nodes[count++] = v;
    }
    layer_sizes[0] = B;

    for (int32_t l = 0; l < L; l++) {
        const int64_t f = fanouts[l];
        const int64_t nd = count;                 /* frontier = every node so far */
        if (rp_used + nd + 1 > cap_rowptr) { rc = ORACLE_CAPACITY; goto done; }
        int32_t* rp = row_ptr + rp_used;
        int64_t e0 = e_used;
        rp[0] = 0;
        pos = (int64_t*)realloc(pos, (size_t)(f > 0 ? f : 1) * sizeof(int64_t));
        for (int64_t r = 0; r < nd; r++) {
            int32_t v = nodes[r];
            int64_t deg = offsets[v + 1] - offsets[v];
            int64_t k = oracle_sample_positions(deg, f, seed, v, m, l, pos);
            if (e_used + k > cap_edges) { rc = ORACLE_CAPACITY; goto done; }
            for (int64_t t = 0; t < k; t++) {
                int32_t u = indices[offsets[v] + pos[t]];
                col[e_used] = u;                  /* global id for now */
                if (col_global) col_global[e_used] = u;
                e_used++;
            }
            rp[r + 1] = (int32_t)(e_used - e0);
        }
        /* union with the minibatch's node set; new nodes ascending */
        if (union_new_sorted(col + e0, e_used - e0, nodes, &count, cap_nodes, id) != 0) {
            rc = ORACLE_CAPACITY;
            goto done;
        }
        /* relabel the hop's columns to local ids */
        for (int64_t e = e0; e < e_used; e++) col[e] = id[col[e]];
        edge_counts[l] = e_used - e0;
        layer_sizes[l + 1] = (int32_t)count;
        rp_used += nd + 1;
    }
done:
    /* restore the scratch map */
    for (int64_t i = 0; i < count; i++) id[nodes[i]] = -1;
    free(pos);
    return rc;
}

/* Gathered feature rows of one node list: out[i] = feat[nodes[i]] (bytes). */
void oracle_gather(const uint8_t* feat, int64_t row_bytes, const int32_t* nodes, int64_t n,
                   uint8_t* out) {
    for (int64_t i = 0; i < n; i++)
        memcpy(out + i * row_bytes, feat + (int64_t)nodes[i] * row_bytes, (size_t)row_bytes);
}

/* ------------------------------------------------------- blocked (Alg. 1) order */

/* Home topology block of v: the block holding the first edge of its adjacency
 * (objects in ascending node order, Sec. 3.2(1)); clamped to the last block. */
static int64_t home_block(const int64_t* offsets, int64_t v, int64_t e_blk, int64_t nblk) {
    int64_t b = offsets[v] / e_blk;
    return b < nblk ? b : nblk - 1;
}

/*
 * The whole hyperbatch in the order of Alg. 1: per hop, bucket the requests of
 * all minibatches by topology block (Bck_{i,j}), visit the non-empty rows of Bck
 * in ascending block order and, inside a row, minibatch by minibatch; then
 * bucket every minibatch's nodes by feature block and gather row by row.
 *
 * Per-minibatch outputs use fixed strides: nodes/features at j*cap_nodes,
 * row_ptr at j*cap_rowptr, col at j*cap_edges; layer_sizes[j*(L+1)+l],
 * edge_counts[j*L+l].  Statistics (exact integers):
 *   stats[0*L+l] requests R_l, stats[1*L+l] sampled edges S_l,
 *   stats[2*L+l] new nodes U_l, stats[3*L+l] non-empty Bck rows T_l,
 *   stats[4*L+0] rows sum |N_j|, stats[4*L+1] distinct rows,
 *   stats[4*L+2] non-empty feature-block rows.
 * Memory: H * num_nodes int32 for the per-minibatch maps (small inputs only).
 */
int oracle_hyperbatch_blocked(int64_t num_nodes, const int64_t* offsets, const int32_t* indices,
                              int64_t block_bytes, const uint8_t* feat, int64_t row_bytes,
                              const int32_t* targets, int32_t H, int32_t B,
                              const int32_t* fanouts, int32_t L, uint64_t seed, int64_t mb_base,
                              int64_t cap_nodes, int32_t* nodes, int32_t* layer_sizes,
                              int64_t* edge_counts, int64_t cap_rowptr, int32_t* row_ptr,
                              int64_t cap_edges, int32_t* col, uint8_t* features,
                              int64_t* stats) {
    const int64_t E = offsets[num_nodes];
    const int64_t e_blk = block_bytes / 4;                  /* int32 edges per block */
    int64_t nblk = (E + e_blk - 1) / e_blk;
    if (nblk < 1) nblk = 1;
    int64_t rpb = block_bytes / row_bytes;                  /* feature rows per block */
    if (rpb < 1) rpb = 1;
    const int64_t nfblk = (num_nodes + rpb - 1) / rpb;

    int rc = ORACLE_OK;
    int32_t* id = (int32_t*)malloc((size_t)H * (size_t)num_nodes * sizeof(int32_t));
    int64_t* count = (int64_t*)calloc((size_t)H, sizeof(int64_t));
    int64_t* rp_used = (int64_t*)calloc((size_t)H, sizeof(int64_t));
    int64_t* e_used = (int64_t*)calloc((size_t)H, sizeof(int64_t));
    int64_t* cell_cnt = NULL;
    int64_t* cell_ptr = NULL;
    int64_t* cell_fill = NULL;
    int64_t* cell_items = NULL;
    int32_t* samp = NULL;
    int32_t* samp_k = NULL;
    int64_t* pos = NULL;
    uint8_t* seen_any = NULL;
    if (!id || !count || !rp_used || !e_used) { rc = ORACLE_NOMEM; goto done; }
    for (int64_t i = 0; i < (int64_t)H * num_nodes; i++) id[i] = -1;
    memset(stats, 0, (size_t)(4 * L + 3) * sizeof(int64_t));

    for (int32_t j = 0; j < H; j++) {
        int32_t* idj = id + (int64_t)j * num_nodes;
        for (int32_t r = 0; r < B; r++) {
            int32_t v = targets[(int64_t)j * B + r];
            if (v < 0 || v >= num_nodes || idj[v] >= 0) { rc = ORACLE_INVALID; goto done; }
            if (count[j] >= cap_nodes) { rc = ORACLE_CAPACITY; goto done; }
            idj[v] = (int32_t)count[j];
            nodes[(int64_t)j * cap_nodes + count[j]++] = v;
        }
        layer_sizes[(int64_t)j * (L + 1)] = B;
    }

    cell_cnt = (int64_t*)calloc((size_t)(nblk * H + 1), sizeof(int64_t));
    cell_ptr = (int64_t*)malloc((size_t)(nblk * H + 1) * sizeof(int64_t));
    cell_fill = (int64_t*)malloc((size_t)(nblk * H + 1) * sizeof(int64_t));
    if (!cell_cnt || !cell_ptr || !cell_fill) { rc = ORACLE_NOMEM; goto done; }

    for (int32_t l = 0; l < L; l++) {
        const int64_t f = fanouts[l];
        /* frontier of minibatch j = its nodes 0..count[j]-1; request index q */
        int64_t R = 0;
        int64_t* qbase = (int64_t*)malloc((size_t)(H + 1) * sizeof(int64_t));
        for (int32_t j = 0; j < H; j++) { qbase[j] = R; R += count[j]; }
        qbase[H] = R;
        stats[0 * L + l] = R;
        /* Bck_{i,j}: the requests of minibatch j whose home block is i */
        memset(cell_cnt, 0, (size_t)(nblk * H + 1) * sizeof(int64_t));
        for (int32_t j = 0; j < H; j++)
            for (int64_t r = 0; r < count[j]; r++) {
                int32_t v = nodes[(int64_t)j * cap_nodes + r];
                cell_cnt[home_block(offsets, v, e_blk, nblk) * H + j]++;
            }
        int64_t s = 0;
        for (int64_t c = 0; c < nblk * H; c++) { cell_ptr[c] = s; cell_fill[c] = s; s += cell_cnt[c]; }
        cell_ptr[nblk * H] = s;
        cell_items = (int64_t*)realloc(cell_items, (size_t)(R > 0 ? R : 1) * sizeof(int64_t));
        for (int32_t j = 0; j < H; j++)
            for (int64_t r = 0; r < count[j]; r++) {
                int32_t v = nodes[(int64_t)j * cap_nodes + r];
                int64_t c = home_block(offsets, v, e_blk, nblk) * H + j;
                cell_items[cell_fill[c]++] = qbase[j] + r;
            }
        /* sampled slots, one per request, filled in block order */
        samp = (int32_t*)realloc(samp, (size_t)(R * f > 0 ? R * f : 1) * sizeof(int32_t));
        samp_k = (int32_t*)realloc(samp_k, (size_t)(R > 0 ? R : 1) * sizeof(int32_t));
        pos = (int64_t*)realloc(pos, (size_t)(f > 0 ? f : 1) * sizeof(int64_t));
        for (int64_t i = 0; i < nblk; i++) {
            if (cell_ptr[i * H + H] == cell_ptr[i * H]) continue;   /* empty Bck row */
            stats[3 * L + l]++;                                     /* one block load */
            for (int32_t j = 0; j < H; j++)
                for (int64_t p = cell_ptr[i * H + j]; p < cell_ptr[i * H + j + 1]; p++) {
                    int64_t q = cell_items[p];
                    int64_t r = q - qbase[j];
                    int32_t v = nodes[(int64_t)j * cap_nodes + r];
                    int64_t deg = offsets[v + 1] - offsets[v];
                    int64_t k = oracle_sample_positions(deg, f, seed, v, mb_base + j, l, pos);
                    for (int64_t t = 0; t < k; t++)
                        samp[q * f + t] = indices[offsets[v] + pos[t]];
                    samp_k[q] = (int32_t)k;
                }
        }
        /* per minibatch: CSR, union with new nodes ascending, relabel */
        for (int32_t j = 0; j < H; j++) {
            int32_t* idj = id + (int64_t)j * num_nodes;
            int32_t* nj = nodes + (int64_t)j * cap_nodes;
            int64_t nd = count[j];
            if (rp_used[j] + nd + 1 > cap_rowptr) { rc = ORACLE_CAPACITY; free(qbase); goto done; }
            int32_t* rp = row_ptr + (int64_t)j * cap_rowptr + rp_used[j];
            int32_t* cj = col + (int64_t)j * cap_edges;
            int64_t e0 = e_used[j];
            rp[0] = 0;
            for (int64_t r = 0; r < nd; r++) {
                int64_t q = qbase[j] + r;
                if (e_used[j] + samp_k[q] > cap_edges) { rc = ORACLE_CAPACITY; free(qbase); goto done; }
                for (int64_t t = 0; t < samp_k[q]; t++) cj[e_used[j]++] = samp[q * f + t];
                rp[r + 1] = (int32_t)(e_used[j] - e0);
            }
            int64_t before = count[j];
            if (union_new_sorted(cj + e0, e_used[j] - e0, nj, &count[j], cap_nodes, idj) != 0) {
                rc = ORACLE_CAPACITY;
                free(qbase);
                goto done;
            }
            int64_t after = count[j];
            for (int64_t e = e0; e < e_used[j]; e++) cj[e] = idj[cj[e]];
            edge_counts[(int64_t)j * L + l] = e_used[j] - e0;
            layer_sizes[(int64_t)j * (L + 1) + l + 1] = (int32_t)after;
            rp_used[j] += nd + 1;
            stats[1 * L + l] += e_used[j] - e0;
            stats[2 * L + l] += after - before;
        }
        free(qbase);
    }

    /* gathering: Bck_{i,j} = nodes of minibatch j in feature block i */
    {
        int64_t ncell = nfblk * H;
        int64_t* gcnt = (int64_t*)calloc((size_t)(ncell + 1), sizeof(int64_t));
        int64_t* gptr = (int64_t*)malloc((size_t)(ncell + 1) * sizeof(int64_t));
        int64_t total = 0;
        for (int32_t j = 0; j < H; j++) total += count[j];
        int64_t* items = (int64_t*)malloc((size_t)(total > 0 ? total : 1) * sizeof(int64_t));
        seen_any = (uint8_t*)calloc((size_t)num_nodes, 1);
        if (!gcnt || !gptr || !items || !seen_any) {
            free(gcnt); free(gptr); free(items); rc = ORACLE_NOMEM; goto done;
        }
        for (int32_t j = 0; j < H; j++)
            for (int64_t i = 0; i < count[j]; i++)
                gcnt[(nodes[(int64_t)j * cap_nodes + i] / rpb) * H + j]++;
        int64_t s = 0;
        for (int64_t c = 0; c < ncell; c++) { gptr[c] = s; s += gcnt[c]; gcnt[c] = gptr[c]; }
        gptr[ncell] = s;
        for (int32_t j = 0; j < H; j++)
            for (int64_t i = 0; i < count[j]; i++) {
                int32_t v = nodes[(int64_t)j * cap_nodes + i];
                items[gcnt[(v / rpb) * H + j]++] = (int64_t)j * cap_nodes + i;
            }
        for (int64_t b = 0; b < nfblk; b++) {
            if (gptr[b * H + H] == gptr[b * H]) continue;           /* empty row */
            stats[4 * L + 2]++;                                     /* one block load */
            for (int32_t j = 0; j < H; j++)
                for (int64_t p = gptr[b * H + j]; p < gptr[b * H + j + 1]; p++) {
                    int64_t slot = items[p];
                    int32_t v = nodes[slot];
                    if (!seen_any[v]) { seen_any[v] = 1; stats[4 * L + 1]++; }
                    memcpy(features + slot * row_bytes, feat + (int64_t)v * row_bytes,
                           (size_t)row_bytes);
                }
        }
        stats[4 * L + 0] = total;
        free(gcnt); free(gptr); free(items);
    }

done:
    free(id); free(count); free(rp_used); free(e_used);
    free(cell_cnt); free(cell_ptr); free(cell_fill); free(cell_items);
    free(samp); free(samp_k); free(pos); free(seen_any);
    return rc;
}

/* ------------------------------------------------------ all cores (CPU baseline) */

/*
 * The plain order on every core: the minibatches of a hyperbatch are
 * independent (each has its own random stream, keyed by its global index), so
 * threads take whole minibatches, each running oracle_minibatch and
 * oracle_gather unchanged on buffers of its own.  Used only to time the CPU
 * baseline; nothing here computes anything the plain functions do not.
 *
 * Per minibatch j the outputs are its layer sizes (layer_sizes[j][L+1]) and
 * edge counts (edge_counts[j][L]); *distinct receives the number of distinct
 * nodes over the hyperbatch (the rows read once by a block-bucketed gather),
 * counted through seen[num_nodes], whose entries must differ from `stamp` on
 * entry.  threads <= 0 leaves the count to the OpenMP runtime; the number used
 * is returned in *used.  Returns ORACLE_OK or the first failing code.
 */
int oracle_hyperbatch_threads(int64_t num_nodes, const int64_t* offsets, const int32_t* indices,
                              const uint8_t* feat, int64_t row_bytes, const int32_t* targets, int32_t H,
                              int32_t B, const int32_t* fanouts, int32_t L, uint64_t seed, int64_t mb_base,
                              int32_t threads, int32_t* layer_sizes, int64_t* edge_counts, uint32_t* seen,
                              uint32_t stamp, int64_t* distinct, int32_t* used) {
    /* per-minibatch capacities, as for one call of oracle_minibatch */
    int64_t cap_n = B, cap_rp = 0, cap_e = 0;
    for (int32_t l = 0; l < L; l++) {
        cap_rp += cap_n + 1;
        cap_e += cap_n * (int64_t)fanouts[l];
        cap_n = cap_n * (1 + (int64_t)fanouts[l]);
        if (cap_n > num_nodes) cap_n = num_nodes;
    }
    if (cap_n < B) cap_n = B;
    int rc_all = ORACLE_OK;
    int64_t nd_all = 0;
    int nthr = 1;
#pragma omp parallel num_threads(threads > 0 ? threads : omp_get_max_threads()) reduction(+ : nd_all)
    {
#pragma omp single
        nthr = omp_get_num_threads();
        int32_t* id = (int32_t*)malloc((size_t)(num_nodes > 0 ? num_nodes : 1) * sizeof(int32_t));
        int32_t* nodes = (int32_t*)malloc((size_t)cap_n * sizeof(int32_t));
        int32_t* rp = (int32_t*)malloc((size_t)(cap_rp > 0 ? cap_rp : 1) * sizeof(int32_t));
        int32_t* col = (int32_t*)malloc((size_t)(cap_e > 0 ? cap_e : 1) * sizeof(int32_t));
        uint8_t* rows = (uint8_t*)malloc((size_t)cap_n * (size_t)row_bytes);
        int ok = id && nodes && rp && col && rows;
        if (ok)
            for (int64_t i = 0; i < num_nodes; i++) id[i] = -1;
#pragma omp for schedule(dynamic, 1)
        for (int32_t j = 0; j < H; j++) {
            if (!ok) {
#pragma omp critical
                rc_all = ORACLE_NOMEM;
                continue;
            }
            int32_t* ls = layer_sizes + (int64_t)j * (L + 1);
            int rc = oracle_minibatch(num_nodes, offsets, indices, targets + (int64_t)j * B, B, fanouts, L, seed,
                                      mb_base + j, cap_n, nodes, ls, edge_counts + (int64_t)j * L, cap_rp, rp,
                                      cap_e, col, NULL, id);
            if (rc != ORACLE_OK) {
#pragma omp critical
                if (rc_all == ORACLE_OK) rc_all = rc;
                continue;
            }
            oracle_gather(feat, row_bytes, nodes, ls[L], rows);
            for (int64_t i = 0; i < ls[L]; i++)
                if (__atomic_exchange_n(&seen[nodes[i]], stamp, __ATOMIC_RELAXED) != stamp) nd_all++;
        }
        free(id); free(nodes); free(rp); free(col); free(rows);
    }
    *distinct = nd_all;
    *used = nthr;
    return rc_all;
}
