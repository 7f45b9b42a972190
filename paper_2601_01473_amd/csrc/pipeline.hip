// The hyperbatch data-preparation pipeline (AGNES, arXiv 2601.01473, Alg. 1) on
// gfx950.
//
// The bucket matrix Bck of Sec. 3.4(3) (rows = blocks, columns = minibatches,
// cells = the nodes a minibatch needs from a block) is kept as one list of all
// (node, minibatch) pairs of the hyperbatch, sorted by node id and then by
// minibatch.  Objects are stored in ascending node order, so a block's row of
// Bck is a contiguous run of this list, and a node needed by several
// minibatches is a run inside it.  Each hop (Alg. 1, sampling loop):
//   k_count     k = min(deg, f_l) per request, in (minibatch, row) order
//   scan        edge offset of every request (the hop's row pointers)
//   k_sample    walks the list in block order: Floyd subsets from Philox words,
//               neighbours written at the request's edge offset
//   radix sort  the sampled neighbours by node id (stable: minibatch order kept)
//   k_heads     runs of equal (node, minibatch); a run is a new node unless the
//               list already holds it (merge-join search)
//   scan        run numbers and new-node numbers
//   k_runs      new nodes in (node, minibatch) order; local ids of old nodes
//   group rank  stable count by minibatch: the rank of a new node among its
//               minibatch's new nodes in id order gives its local id
//   k_relabel   hop columns in local ids
//   k_merge     new (node, minibatch) pairs merged into the sorted list
// Gather (Alg. 1, gathering loop): the final list is the feature bucket in block
// order; k_gather copies each row to every minibatch that needs it.
//
// Nothing here uses a device-wide atomic per element; every size stays on the
// device until one synchronisation before the gather.
#include <algorithm>
#include <cstring>

#include "device.hpp"
#include "runtime.hpp"

namespace agnes {

struct Geometry {
    int32_t H, B, L;
    int64_t capN;                      // node capacity of one minibatch
    int64_t cap[AGNES_MAX_LAYERS + 1]; // cap[l] = frontier capacity of hop l (cap[L] = capN)
    int64_t Rmax, Smax, rows_max, sort_max;
    int jbits;
};

static Geometry plan(const Store& s, int32_t H, int32_t B, const int32_t* fanouts, int32_t L) {
    Geometry g{};
    g.H = H; g.B = B; g.L = L;
    g.cap[0] = B;
    g.Rmax = 0; g.Smax = 0;
    const int64_t nmax = std::max<int64_t>(s.num_nodes, B);
    for (int l = 0; l < L; l++) {
        g.Rmax = std::max<int64_t>(g.Rmax, (int64_t)H * g.cap[l]);
        g.Smax = std::max<int64_t>(g.Smax, (int64_t)H * g.cap[l] * fanouts[l]);
        g.cap[l + 1] = std::min<int64_t>(g.cap[l] * (1 + (int64_t)fanouts[l]), nmax);
    }
    g.capN = g.cap[L];
    g.rows_max = (int64_t)H * g.capN;
    g.sort_max = std::max<int64_t>(g.Smax, (int64_t)H * B);
    int jb = 0;
    while ((1 << jb) < H) jb++;
    g.jbits = jb;
    return g;
}

constexpr int kGroupWGs = 512;          // workgroups of the by-minibatch counting pass
constexpr int kSortTileR = 2048;        // entries per tile of the by-minibatch ranking

// ----------------------------------------------------------------- small kernels

__device__ __forceinline__ void load_offsets(int64_t* dst, const int64_t* src, int n) {
    for (int i = threadIdx.x; i <= n; i += kBlock) dst[i] = src[i];
    __syncthreads();
}

// Minibatch of edge e given the request offsets: mb_e[j] = e_off[req_off[j]].
__device__ __forceinline__ void load_mb_edges(int64_t* mb_e, const int64_t* req_off, const int64_t* e_off, int H) {
    for (int i = threadIdx.x; i <= H; i += kBlock) mb_e[i] = e_off[req_off[i]];
    __syncthreads();
}

__global__ void k_ctl_init(Ctl* ctl, int64_t targets) {
    int64_t* p = (int64_t*)ctl;
    for (int i = threadIdx.x; i < (int)(sizeof(Ctl) / 8); i += kBlock) p[i] = 0;
    __syncthreads();
    if (threadIdx.x == 0) ctl->targets = targets;
}

// Targets become the first B nodes of every minibatch.  An out-of-range target
// is recorded as an error and replaced by node 0 so that later kernels stay in
// bounds.  tkey receives the node ids for the sort that builds the list.
__global__ __launch_bounds__(kBlock) void k_init(const int32_t* targets, int H, int B, int64_t num_nodes,
                                                 int64_t capN, int32_t* nodes, int32_t* size,
                                                 int64_t* newcnt, uint32_t* tkey, Ctl* ctl) {
    int64_t n = (int64_t)H * B;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += (int64_t)gridDim.x * kBlock) {
        int64_t j = i / B, r = i - j * B;
        int32_t v = targets[i];
        if (v < 0 || v >= num_nodes) {
            atomicOr((unsigned long long*)&ctl->err, 1ull);
            v = 0;
        }
        nodes[j * capN + r] = v;
        tkey[i] = (uint32_t)v;
        if (r == 0) {
            size[j] = B;
            newcnt[j] = 0;
        }
    }
}

// The list of hop 0: targets sorted by (node, minibatch), value = row r.  Equal
// neighbours with the same minibatch are duplicate targets.
__global__ __launch_bounds__(kBlock) void k_list0(const uint32_t* sk, const uint32_t* sv, int B,
                                                  uint64_t* rl_key, int32_t* rl_val, Ctl* ctl) {
    const int64_t n = ctl->targets;
    for (int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x; p < n; p += (int64_t)gridDim.x * kBlock) {
        uint32_t u = sk[p];
        uint32_t i = sv[p];
        uint32_t j = i / (uint32_t)B, r = i - j * (uint32_t)B;
        rl_key[p] = ((uint64_t)u << 32) | j;
        rl_val[p] = (int32_t)r;
        if (p > 0 && sk[p - 1] == u && sv[p - 1] / (uint32_t)B == j)
            atomicOr((unsigned long long*)&ctl->err, 2ull);
    }
}

// Block 0: per-minibatch bookkeeping between hops.  Entering hop l (l < L) it
// closes hop l-1 (edge counts, node counts grown by the new nodes) and computes
// the request offsets of hop l; with l == L it closes the last hop and computes
// the output row offsets.
__global__ __launch_bounds__(kBlock) void k_begin(int l, int L, int H, Ctl* ctl, int32_t* size,
                                                  int64_t* newcnt, int32_t* lsz, int64_t* ecount,
                                                  int64_t* req_off, const int64_t* e_off, int64_t* node_off) {
    __shared__ int64_t lds[kWavesPerBlock];
    if (l > 0) {
        for (int j = threadIdx.x; j < H; j += kBlock) {
            ecount[(int64_t)j * L + (l - 1)] = e_off[req_off[j + 1]] - e_off[req_off[j]];
            size[j] += (int32_t)newcnt[j];
            newcnt[j] = 0;
        }
        if (threadIdx.x == 0) {
            ctl->sampled[l - 1] = ctl->S;
            ctl->new_nodes[l - 1] = ctl->n_new;
        }
        __syncthreads();
    }
    int64_t* out = (l < L) ? req_off : node_off;
    int64_t carry = 0;
    for (int base = 0; base < H; base += kBlock) {
        int j = base + threadIdx.x;
        int64_t v = (j < H) ? size[j] : 0;
        if (j < H) lsz[(int64_t)j * (L + 1) + l] = (int32_t)v;
        int64_t total;
        int64_t ex = block_exclusive_scan(v, lds, total);
        if (j < H) out[j] = carry + ex;
        carry += total;
    }
    if (threadIdx.x == 0) {
        out[H] = carry;
        if (l < L) {
            ctl->R = carry;
            ctl->requests[l] = carry;
            ctl->n_new = 0;
            ctl->S = 0;
        } else {
            ctl->rows = carry;
        }
    }
}

// ----------------------------------------------------------------- sampling

template <typename OffT>
__global__ __launch_bounds__(kBlock) void k_count(int H, int64_t capN, int32_t f, const OffT* off,
                                                  const int32_t* nodes, const int64_t* req_off_g,
                                                  int32_t* cnt, const Ctl* ctl) {
    extern __shared__ int64_t req_off[];
    load_offsets(req_off, req_off_g, H);
    const int64_t R = ctl->R;
    for (int64_t q = (int64_t)blockIdx.x * kBlock + threadIdx.x; q < R; q += (int64_t)gridDim.x * kBlock) {
        int j = upper_segment(req_off, H, q);
        int32_t v = nodes[(int64_t)j * capN + (q - req_off[j])];
        int64_t deg = (int64_t)off[v + 1] - (int64_t)off[v];
        cnt[q] = (int32_t)(deg < f ? deg : f);
    }
}

// Sample every request of the hop, walking the list in (node, minibatch) order:
// consecutive threads serve the requests of the same topology block from every
// minibatch, and the requests of one node are neighbours.  Also counts the
// topology blocks the hop touches (non-empty rows of Bck).
template <typename OffT, int MAXK>
__global__ __launch_bounds__(kBlock) void k_sample(int l, int H, int32_t f, uint64_t seed, int64_t mb_base,
                                                   const OffT* off, const int32_t* adj, int e_blk_log2,
                                                   int64_t nblk, const uint64_t* rl_key, const int32_t* rl_val,
                                                   const int64_t* req_off_g, const int64_t* e_off,
                                                   int32_t* cg, int32_t* row_ptr,
                                                   Ctl* ctl) {
    extern __shared__ int64_t req_off[];      // [H+1] request offsets, then [H+1] edge offsets
    int64_t* mb_e = req_off + (H + 1);
    for (int i = threadIdx.x; i <= H; i += kBlock) {
        int64_t ro = req_off_g[i];
        req_off[i] = ro;
        mb_e[i] = e_off[ro];
    }
    __syncthreads();
    const int64_t R = ctl->R;
    for (int64_t base = (int64_t)blockIdx.x * kBlock; base < R; base += (int64_t)gridDim.x * kBlock) {
        int64_t p = base + threadIdx.x;
        bool active = p < R;
        int64_t blk = -1;
        if (active) {
            uint64_t key = rl_key[p];
            int32_t v = (int32_t)(key >> 32);
            int j = (int)(uint32_t)key;
            int64_t r = rl_val[p];
            int64_t q = req_off[j] + r;
            int64_t o0 = (int64_t)off[v];
            int64_t deg = (int64_t)off[v + 1] - o0;
            blk = o0 >> e_blk_log2;
            if (blk >= nblk) blk = nblk - 1;
            int k = (int)(deg < f ? deg : f);
            int64_t eo = e_off[q];
            int64_t mb_e0 = mb_e[j];
            int32_t* out = cg + eo;
            const int32_t* a = adj + o0;
            if (k == deg) {
                for (int t = 0; t < k; t++) out[t] = a[t];
            } else if (MAXK > 0) {
                floyd_sample_regs<(MAXK > 0 ? MAXK : 1)>((uint64_t)deg, k, seed, (uint64_t)v,
                                                         (uint64_t)(mb_base + j), (uint64_t)l, a, out);
            } else {
                floyd_sample_mem((uint64_t)deg, k, seed, (uint64_t)v, (uint64_t)(mb_base + j), (uint64_t)l, a, out);
            }
            int64_t rp = req_off[j] + j + r;
            row_ptr[rp] = (int32_t)(eo - mb_e0);
            if (q + 1 == req_off[j + 1]) row_ptr[rp + 1] = (int32_t)(eo + k - mb_e0);
        }
        // a request opens a new Bck row when its block differs from the previous request's
        int64_t prev = (int64_t)shfl64((uint64_t)blk, lane_id() > 0 ? lane_id() - 1 : 0);
        if (lane_id() == 0 && active && p > 0) {
            int32_t vp = (int32_t)(rl_key[p - 1] >> 32);
            prev = (int64_t)off[vp] >> e_blk_log2;
            if (prev >= nblk) prev = nblk - 1;
        }
        bool opens = active && (p == 0 || prev != blk);
        uint64_t m = __ballot(opens);
        if (lane_id() == 0 && m) atomicAdd((unsigned long long*)&ctl->topo_blocks[l], (unsigned long long)__popcll(m));
    }
}

// Runs of the sorted sampled neighbours.  For sorted edge p: (u, j) = (node,
// minibatch of the edge); a run head is the first edge of a (u, j) pair.  A head
// looks its pair up in the list (sorted the same way): found = an old node with
// local id hl[p]; not found = a new node.  pk[p] = (head << 32) | new.
// Each workgroup takes tiles of 2048 sorted edges, narrows the list to the key
// range of the tile with two searches and stages that range in LDS.
constexpr int kHeadTile = 2048;
constexpr int kHeadCap = 2048;

__global__ __launch_bounds__(kBlock) void k_heads(int H, const int64_t* req_off, const int64_t* e_off,
                                                  const uint32_t* su, const uint32_t* se,
                                                  const uint64_t* rl_key, const int32_t* rl_val,
                                                  int64_t* pk, int32_t* hl, const Ctl* ctl) {
    extern __shared__ int64_t mb_e[];
    __shared__ uint64_t tk[kHeadTile];
    __shared__ uint64_t lk[kHeadCap];
    __shared__ int32_t lv[kHeadCap];
    __shared__ int64_t range[2];
    __shared__ uint64_t prevk;
    load_mb_edges(mb_e, req_off, e_off, H);
    const int t = threadIdx.x;
    const int64_t S = ctl->S, R = ctl->R;
    for (int64_t t0 = (int64_t)blockIdx.x * kHeadTile; t0 < S; t0 += (int64_t)gridDim.x * kHeadTile) {
        const int cnt = (int)((S - t0) < kHeadTile ? (S - t0) : kHeadTile);
        for (int i = t; i < cnt; i += kBlock)
            tk[i] = ((uint64_t)su[t0 + i] << 32) | (uint32_t)upper_segment(mb_e, H, (int64_t)se[t0 + i]);
        if (t == 0)
            prevk = t0 > 0 ? (((uint64_t)su[t0 - 1] << 32) | (uint32_t)upper_segment(mb_e, H, (int64_t)se[t0 - 1]))
                           : ~0ull;
        __syncthreads();
        {
            // the list range holding the tile's keys: [lower_bound(first), upper_bound(last))
            const uint64_t kf = tk[0], kl = tk[cnt - 1];
            const int64_t a = block_partition_point(0, R, [&](int64_t i) { return rl_key[i] < kf; });
            const int64_t b = block_partition_point(a, R, [&](int64_t i) { return rl_key[i] <= kl; });
            if (t == 0) { range[0] = a; range[1] = b; }
        }
        __syncthreads();
        const int64_t lo = range[0], hi = range[1];
        const int64_t m = hi - lo;
        const bool staged = m <= kHeadCap;
        if (staged)
            for (int i = t; i < m; i += kBlock) {
                lk[i] = rl_key[lo + i];
                lv[i] = rl_val[lo + i];
            }
        __syncthreads();
        for (int i = t; i < cnt; i += kBlock) {
            const uint64_t key = tk[i];
            const bool head = key != (i > 0 ? tk[i - 1] : prevk);
            bool found = false;
            int32_t local = -1;
            if (head) {
                if (staged) {
                    int a = 0, b = (int)m;
                    while (a < b) {
                        int mid = (a + b) >> 1;
                        if (lk[mid] < key) a = mid + 1; else b = mid;
                    }
                    if (a < m && lk[a] == key) { found = true; local = lv[a]; }
                } else {
                    int64_t a = lo, b = hi;
                    while (a < b) {
                        int64_t mid = (a + b) >> 1;
                        if (rl_key[mid] < key) a = mid + 1; else b = mid;
                    }
                    if (a < hi && rl_key[a] == key) { found = true; local = rl_val[a]; }
                }
            }
            pk[t0 + i] = ((int64_t)(head ? 1 : 0) << 32) | (int64_t)((head && !found) ? 1 : 0);
            hl[t0 + i] = local;
        }
        __syncthreads();
    }
}

// Heads of new pairs go to the new-node list (in (node, minibatch) order) with
// their run number; heads of old pairs give their run its local id.
__global__ __launch_bounds__(kBlock) void k_runs(int H, const int64_t* req_off, const int64_t* e_off,
                                                 const uint32_t* su, const uint32_t* se, const int64_t* pk,
                                                 const int64_t* pkx, const int32_t* hl, uint64_t* nl_key,
                                                 int32_t* nl_run, int32_t* run_local, Ctl* ctl) {
    extern __shared__ int64_t mb_e[];
    load_mb_edges(mb_e, req_off, e_off, H);
    const int64_t S = ctl->S;
    if (blockIdx.x == 0 && threadIdx.x == 0) ctl->n_new = ctl->pktot & 0xFFFFFFFFll;
    for (int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x; p < S; p += (int64_t)gridDim.x * kBlock) {
        int64_t f = pk[p];
        if (!(f >> 32)) continue;
        int64_t x = pkx[p];
        int32_t run = (int32_t)(x >> 32);
        if (f & 1) {
            int64_t ni = x & 0xFFFFFFFFll;
            nl_key[ni] = ((uint64_t)su[p] << 32) | (uint32_t)upper_segment(mb_e, H, (int64_t)se[p]);
            nl_run[ni] = run;
        } else {
            run_local[run] = hl[p];
        }
    }
}

__device__ __forceinline__ void group_range(int64_t n, int g, int64_t& lo, int64_t& hi) {
    int64_t chunk = (n + kGroupWGs - 1) / kGroupWGs;
    lo = (int64_t)g * chunk;
    if (lo > n) lo = n;
    hi = lo + chunk;
    if (hi > n) hi = n;
}

// Per workgroup range of the new-node list: how many new nodes each minibatch has.
__global__ __launch_bounds__(kBlock) void k_grp_hist(const uint64_t* nl_key, int H, int64_t* ghist,
                                                     const Ctl* ctl) {
    extern __shared__ uint32_t h[];
    for (int j = threadIdx.x; j < H; j += kBlock) h[j] = 0;
    __syncthreads();
    int64_t lo, hi;
    group_range(ctl->n_new, blockIdx.x, lo, hi);
    for (int64_t i = lo + threadIdx.x; i < hi; i += kBlock) atomicAdd(&h[(uint32_t)nl_key[i]], 1u);
    __syncthreads();
    for (int j = threadIdx.x; j < H; j += kBlock) ghist[(int64_t)j * kGroupWGs + blockIdx.x] = h[j];
}

// Per minibatch j (one workgroup each): offsets of each workgroup's range; the
// minibatch's new-node count.
__global__ __launch_bounds__(kBlock) void k_grp_scan(int64_t* ghist, int64_t* newcnt) {
    __shared__ int64_t lds[kWavesPerBlock];
    int64_t* row = ghist + (int64_t)blockIdx.x * kGroupWGs;
    constexpr int per = kGroupWGs / kBlock;
    int64_t v[per];
    int64_t local = 0;
#pragma unroll
    for (int k = 0; k < per; k++) {
        v[k] = row[threadIdx.x * per + k];
        local += v[k];
    }
    int64_t total;
    int64_t ex = block_exclusive_scan(local, lds, total);
#pragma unroll
    for (int k = 0; k < per; k++) {
        row[threadIdx.x * per + k] = ex;
        ex += v[k];
    }
    if (threadIdx.x == 0) newcnt[blockIdx.x] = total;
}

// Stable rank of each new node among the new nodes of its minibatch (the list
// is in id order within a minibatch): local id = |S_{j,l-1}| + rank.  A
// workgroup walks its range in tiles of 2048: wave w counts its 512 entries per
// minibatch with ballots (lane order, then round order), the waves' counts are
// stacked per minibatch (wave order), then every entry gets its local id.
// Dynamic LDS: H int64 cursors + 4 x H int32 counts.
__global__ __launch_bounds__(kBlock) void k_grp_rank(const uint64_t* nl_key, const int32_t* nl_run, int H,
                                                     int jbits, const int64_t* ghist, const int32_t* size,
                                                     int64_t capN, int32_t* nodes, int32_t* run_local,
                                                     int32_t* nl_val, Ctl* ctl) {
    extern __shared__ int64_t cursor[];
    int32_t* wc = (int32_t*)(cursor + H);           // [kWavesPerBlock][H]
    const int t = threadIdx.x, w = wave_id(), lane = lane_id();
    for (int j = t; j < H; j += kBlock) cursor[j] = ghist[(int64_t)j * kGroupWGs + blockIdx.x] + size[j];
    int64_t lo, hi;
    group_range(ctl->n_new, blockIdx.x, lo, hi);
    for (int64_t t0 = lo; t0 < hi; t0 += kSortTileR) {
        for (int x = t; x < kWavesPerBlock * H; x += kBlock) wc[x] = 0;
        __syncthreads();
        int jr[8], rk[8];
#pragma unroll
        for (int r = 0; r < 8; r++) {
            const int64_t i = t0 + w * 512 + r * kWave + lane;
            const bool valid = i < hi;
            const int j = valid ? (int)(uint32_t)nl_key[i] : 0;
            uint64_t peers = __ballot(valid);
            for (int b = 0; b < jbits; b++) {
                uint64_t m = __ballot((j >> b) & 1);
                peers &= ((j >> b) & 1) ? m : ~m;
            }
            const int rank = __popcll(peers & lanemask_lt());
            const int leader = valid ? (__ffsll((unsigned long long)peers) - 1) : lane;
            int old = 0;
            if (valid && rank == 0) {
                old = wc[w * H + j];
                wc[w * H + j] = old + __popcll(peers);
            }
            old = __shfl(old, leader, kWave);
            jr[r] = valid ? j : -1;
            rk[r] = old + rank;
        }
        __syncthreads();
        for (int j = t; j < H; j += kBlock) {
            int64_t c = cursor[j];
            for (int ww = 0; ww < kWavesPerBlock; ww++) {
                int n = wc[ww * H + j];
                wc[ww * H + j] = (int32_t)c;
                c += n;
            }
            cursor[j] = c;
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < 8; r++) {
            if (jr[r] < 0) continue;
            const int64_t i = t0 + w * 512 + r * kWave + lane;
            const int j = jr[r];
            const int64_t local = (int64_t)wc[w * H + j] + rk[r];
            if (local >= capN) {
                atomicOr((unsigned long long*)&ctl->err, 4ull);
            } else {
                nodes[(int64_t)j * capN + local] = (int32_t)(nl_key[i] >> 32);
                run_local[nl_run[i]] = (int32_t)local;
                nl_val[i] = (int32_t)local;
            }
        }
        __syncthreads();
    }
}

// Every sampled edge takes the local id of its run.
__global__ __launch_bounds__(kBlock) void k_relabel(const int64_t* pk, const int64_t* pkx, const uint32_t* se,
                                                    const int32_t* run_local, int32_t* col, const Ctl* ctl) {
    const int64_t S = ctl->S;
    for (int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x; p < S; p += (int64_t)gridDim.x * kBlock) {
        int32_t run = (int32_t)((pkx[p] + pk[p]) >> 32) - 1;
        col[se[p]] = run_local[run];
    }
}

// Merge of the list (R pairs) with the hop's new pairs (n_new), both sorted and
// disjoint, by merge path: a workgroup takes 2048 outputs, finds where they
// start and end on the two inputs (two searches), stages both pieces in LDS and
// every thread merges 8 outputs after a local search.
constexpr int kMergeTile = 2048;
constexpr int kMergeItems = kMergeTile / kBlock;

__global__ __launch_bounds__(kBlock) void k_merge(const uint64_t* ak, const int32_t* av, const uint64_t* bk,
                                                  const int32_t* bv, uint64_t* ck, int32_t* cv, const Ctl* ctl) {
    __shared__ uint64_t sk[kMergeTile];
    __shared__ int32_t sv[kMergeTile];
    __shared__ int64_t split[2];
    const int t = threadIdx.x;
    const int64_t na = ctl->R, nb = ctl->n_new, n = na + nb;
    for (int64_t d0 = (int64_t)blockIdx.x * kMergeTile; d0 < n; d0 += (int64_t)gridDim.x * kMergeTile) {
        const int64_t d1 = (n - d0) < kMergeTile ? n : d0 + kMergeTile;
        if (t < 2) {
            // merge path: number of A elements among the first d outputs
            const int64_t d = t == 0 ? d0 : d1;
            int64_t lo = d > nb ? d - nb : 0, hi = d < na ? d : na;
            while (lo < hi) {
                int64_t mid = (lo + hi) >> 1;
                if (ak[mid] < bk[d - 1 - mid]) lo = mid + 1; else hi = mid;
            }
            split[t] = lo;
        }
        __syncthreads();
        const int64_t a0 = split[0], a1 = split[1];
        const int64_t b0 = d0 - a0, b1 = d1 - a1;
        const int nA = (int)(a1 - a0), nB = (int)(b1 - b0);
        for (int i = t; i < nA; i += kBlock) { sk[i] = ak[a0 + i]; sv[i] = av[a0 + i]; }
        for (int i = t; i < nB; i += kBlock) { sk[nA + i] = bk[b0 + i]; sv[nA + i] = bv[b0 + i]; }
        __syncthreads();
        const int dl = t * kMergeItems;
        const int total = nA + nB;
        if (dl < total) {
            int lo = dl > nB ? dl - nB : 0, hi = dl < nA ? dl : nA;
            while (lo < hi) {
                int mid = (lo + hi) >> 1;
                if (sk[mid] < sk[nA + dl - 1 - mid]) lo = mid + 1; else hi = mid;
            }
            int ai = lo, bi = dl - lo;
            for (int k = 0; k < kMergeItems && dl + k < total; k++) {
                const bool takea = bi >= nB || (ai < nA && sk[ai] < sk[nA + bi]);
                const int src = takea ? ai++ : nA + bi++;
                ck[d0 + dl + k] = sk[src];
                cv[d0 + dl + k] = sv[src];
            }
        }
        __syncthreads();
    }
}

// ----------------------------------------------------------------- gather

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Row copy over the final list, which is the feature bucket of Alg. 1's
// gathering loop in block order: the requests of a feature block are contiguous
// and those of one node are neighbours, so each row is loaded from HBM once and
// written to every minibatch that needs it (dest = node_off[j] + local id).
// LPR lanes share a row (16-byte or 4-byte units).  Each lane group loads the
// keys of U rows, then U row pieces, then stores them, so U rows are in flight
// per group.  Workgroup b takes a contiguous range; ranges are dealt so that
// neighbouring ranges (the same blocks) run on the same XCD.  Also counts the
// distinct rows and the non-empty feature-block rows.
template <typename Unit, int LPR, int U>
__global__ __launch_bounds__(kBlock) void k_gather(const Unit* __restrict__ feat, Unit* __restrict__ out,
                                                   int32_t* __restrict__ nodes_out,
                                                   const uint64_t* __restrict__ rl_key,
                                                   const int32_t* __restrict__ rl_val, const int64_t* node_off_g,
                                                   int H, int64_t rows, int64_t row_units, uint32_t rpb,
                                                   Ctl* ctl) {
    constexpr int RPW = kWave / LPR;             // lane groups (rows) per wave
    constexpr int GPB = kWavesPerBlock * RPW;    // lane groups per workgroup
    extern __shared__ int64_t node_off[];
    __shared__ unsigned long long cnt[2];
    if (threadIdx.x < 2) cnt[threadIdx.x] = 0;
    load_offsets(node_off, node_off_g, H);
    const int G = gridDim.x;
    const int b = blockIdx.x;
    const int lb = (G % 8 == 0) ? (b % 8) * (G / 8) + b / 8 : b;
    const int64_t chunk = (rows + G - 1) / G;
    const int64_t lo = std::min<int64_t>(rows, (int64_t)lb * chunk);
    const int64_t hi = std::min<int64_t>(rows, lo + chunk);
    const int li = lane_id() % LPR;
    const int gid = wave_id() * RPW + lane_id() / LPR;
    unsigned long long nd = 0, nf = 0;
    for (int64_t e0 = lo + gid; e0 < hi; e0 += (int64_t)GPB * U) {
        int64_t src[U], dst[U];
        bool ok[U];
#pragma unroll
        for (int k = 0; k < U; k++) {
            const int64_t e = e0 + (int64_t)k * GPB;
            ok[k] = e < hi;
            src[k] = 0;
            dst[k] = 0;
            if (ok[k]) {
                const uint64_t key = rl_key[e];
                const uint32_t u = (uint32_t)(key >> 32);
                src[k] = (int64_t)u * row_units;
                const int64_t d = node_off[(uint32_t)key] + rl_val[e];
                dst[k] = d * row_units;
                if (li == 0) {
                    nodes_out[d] = (int32_t)u;
                    const uint32_t pu = e > 0 ? (uint32_t)(rl_key[e - 1] >> 32) : 0xFFFFFFFFu;
                    nd += (pu != u);
                    nf += (e == 0 || pu / rpb != u / rpb);
                }
            }
        }
        for (int64_t c = li; c < row_units; c += LPR) {
            Unit x[U];
#pragma unroll
            for (int k = 0; k < U; k++)
                if (ok[k]) x[k] = feat[src[k] + c];
#pragma unroll
            for (int k = 0; k < U; k++)
                if (ok[k]) __builtin_nontemporal_store(x[k], out + dst[k] + c);
        }
    }
    if (nd) atomicAdd(&cnt[0], nd);
    if (nf) atomicAdd(&cnt[1], nf);
    __syncthreads();
    if (threadIdx.x == 0) {
        if (cnt[0]) atomicAdd((unsigned long long*)&ctl->distinct, cnt[0]);
        if (cnt[1]) atomicAdd((unsigned long long*)&ctl->fblocks, cnt[1]);
    }
}

template <typename Unit, int LPR>
static void launch_gather_u(int unroll, dim3 grid, size_t lds, hipStream_t st, const Unit* f, Unit* o,
                            int32_t* nodes_out, const uint64_t* rl_key, const int32_t* rl_val,
                            const int64_t* node_off, int H, int64_t rows, int64_t row_units, uint32_t rpb,
                            Ctl* ctl) {
    if (unroll >= 8)
        hipLaunchKernelGGL((k_gather<Unit, LPR, 8>), grid, dim3(kBlock), lds, st, f, o, nodes_out, rl_key, rl_val,
                           node_off, H, rows, row_units, rpb, ctl);
    else if (unroll >= 4)
        hipLaunchKernelGGL((k_gather<Unit, LPR, 4>), grid, dim3(kBlock), lds, st, f, o, nodes_out, rl_key, rl_val,
                           node_off, H, rows, row_units, rpb, ctl);
    else
        hipLaunchKernelGGL((k_gather<Unit, LPR, 2>), grid, dim3(kBlock), lds, st, f, o, nodes_out, rl_key, rl_val,
                           node_off, H, rows, row_units, rpb, ctl);
}

template <typename Unit>
static void launch_gather(const void* feat, void* out, int32_t* nodes_out, const uint64_t* rl_key,
                          const int32_t* rl_val, const int64_t* node_off, int H, int64_t rows,
                          int64_t row_units, uint32_t rpb, Ctl* ctl, int groups, int unroll, hipStream_t st) {
    int G = grid_for(rows * row_units / 64 + 1, groups);
    G = std::max(8, (G + 7) / 8 * 8);
    const Unit* f = (const Unit*)feat;
    Unit* o = (Unit*)out;
    const size_t lds = (size_t)(H + 1) * sizeof(int64_t);
    const dim3 grid(G);
    if (row_units >= 64)
        launch_gather_u<Unit, 64>(unroll, grid, lds, st, f, o, nodes_out, rl_key, rl_val, node_off, H, rows, row_units, rpb, ctl);
    else if (row_units > 16)
        launch_gather_u<Unit, 32>(unroll, grid, lds, st, f, o, nodes_out, rl_key, rl_val, node_off, H, rows, row_units, rpb, ctl);
    else if (row_units > 8)
        launch_gather_u<Unit, 16>(unroll, grid, lds, st, f, o, nodes_out, rl_key, rl_val, node_off, H, rows, row_units, rpb, ctl);
    else if (row_units > 4)
        launch_gather_u<Unit, 8>(unroll, grid, lds, st, f, o, nodes_out, rl_key, rl_val, node_off, H, rows, row_units, rpb, ctl);
    else
        launch_gather_u<Unit, 4>(unroll, grid, lds, st, f, o, nodes_out, rl_key, rl_val, node_off, H, rows, row_units, rpb, ctl);
}

// ----------------------------------------------------------------- host orchestration

// Layout of the block that the host reads at the synchronisation point:
// [Ctl][layer sizes H x (L+1) int32][edge counts H x L int64].
struct SyncLayout {
    size_t lsz, ecount, bytes;
};

static SyncLayout sync_layout(int H, int L) {
    SyncLayout y;
    y.lsz = (sizeof(Ctl) + 255) / 256 * 256;
    y.ecount = (y.lsz + (size_t)H * (L + 1) * 4 + 255) / 256 * 256;
    y.bytes = y.ecount + (size_t)H * L * 8;
    return y;
}

static void reserve_workspace(Workspace& w, const Geometry& g, const SyncLayout& y) {
    const int64_t H = g.H;
    w.nodes.reserve((size_t)g.rows_max * 4);
    w.size.reserve((size_t)H * 4);
    w.newcnt.reserve((size_t)H * 8);
    w.req_off.reserve((size_t)(H + 1) * 8);
    w.mb_off.reserve((size_t)(H + 1) * 8);
    w.sync.reserve(y.bytes);
    w.sync_host.reserve(y.bytes);
    w.cnt.reserve((size_t)g.Rmax * 4);
    w.e_off.reserve((size_t)(g.Rmax + 1) * 8);
    for (int i = 0; i < 2; i++) {
        w.rl_key[i].reserve((size_t)g.rows_max * 8);
        w.rl_val[i].reserve((size_t)g.rows_max * 4);
    }
    w.skey.reserve((size_t)g.sort_max * 4);
    w.sval.reserve((size_t)g.sort_max * 4);
    w.skey2.reserve((size_t)g.sort_max * 4);
    w.sval2.reserve((size_t)g.sort_max * 4);
    w.pk.reserve((size_t)g.Smax * 8);
    w.pkx.reserve((size_t)(g.Smax + 1) * 8);
    w.hl.reserve((size_t)g.Smax * 4);
    w.nl_key.reserve((size_t)g.Smax * 8);
    w.nl_run.reserve((size_t)g.Smax * 4);
    w.nl_val.reserve((size_t)g.Smax * 4);
    w.run_local.reserve((size_t)g.Smax * 4);
    w.ghist.reserve((size_t)H * kGroupWGs * 8);
    w.rs_hist.reserve((size_t)radix_hist_entries(g.sort_max) * 4);
    w.rs_dtot.reserve((size_t)radix_dtot_entries() * 4);
    w.scan_part.reserve((size_t)scan_partials_needed() * 8);
    if (!w.ev[0])
        for (auto& e : w.ev) AGNES_CHECK_HIP(hipEventCreate(&e));
}

template <typename OffT>
static void launch_layer(const Store& s, Workspace& w, const Geometry& g, int l, int32_t f, uint64_t seed,
                         int64_t mb_base, Batch& b, const SyncLayout& y, int cur, hipStream_t st) {
    Ctl* ctl = w.sync.as<Ctl>();
    int32_t* lsz = (int32_t*)((char*)w.sync.ptr + y.lsz);
    int64_t* ecount = (int64_t*)((char*)w.sync.ptr + y.ecount);
    const OffT* off = s.offsets.as<OffT>();
    const size_t lds_h = (size_t)(g.H + 1) * sizeof(int64_t);
    const int gR = grid_for(g.Rmax, 2048);
    const int gS = grid_for(g.Smax, 4096);
    int64_t* part = w.scan_part.as<int64_t>();
    const uint64_t* rlk = w.rl_key[cur].as<uint64_t>();
    const int32_t* rlv = w.rl_val[cur].as<int32_t>();

    hipLaunchKernelGGL(k_begin, dim3(1), dim3(kBlock), 0, st, l, g.L, g.H, ctl, w.size.as<int32_t>(),
                       w.newcnt.as<int64_t>(), lsz, ecount, w.req_off.as<int64_t>(), w.e_off.as<int64_t>(),
                       (int64_t*)nullptr);
    hipLaunchKernelGGL(k_count<OffT>, dim3(gR), dim3(kBlock), lds_h, st, g.H, g.capN, f, off,
                       w.nodes.as<int32_t>(), w.req_off.as<int64_t>(), w.cnt.as<int32_t>(), ctl);
    scan_counts(w.cnt.as<int32_t>(), w.e_off.as<int64_t>(), &ctl->R, g.Rmax, &ctl->S, part, st);
    int32_t* rp = b.row_ptr[l].as<int32_t>();
    const int32_t* adj = s.indices.as<int32_t>();
    int32_t* cg = w.skey.as<int32_t>();
#define AGNES_SAMPLE(MK)                                                                               \
    hipLaunchKernelGGL((k_sample<OffT, MK>), dim3(gR), dim3(kBlock), 2 * lds_h, st, l, g.H, f, seed,     \
                       mb_base, off, adj, s.e_blk_log2, s.nblk, rlk, rlv, w.req_off.as<int64_t>(),      \
                       w.e_off.as<int64_t>(), cg, rp, ctl)
    if (f <= 4) AGNES_SAMPLE(4);
    else if (f <= 8) AGNES_SAMPLE(8);
    else if (f <= 16) AGNES_SAMPLE(16);
    else if (f <= 32) AGNES_SAMPLE(32);
    else AGNES_SAMPLE(0);
#undef AGNES_SAMPLE
    // sampled neighbours sorted by node id; values = edge numbers (stable: minibatch order kept)
    int in_tmp = radix_sort_pairs32(w.skey.as<uint32_t>(), w.sval.as<uint32_t>(), w.skey2.as<uint32_t>(),
                                    w.sval2.as<uint32_t>(), &ctl->S, g.Smax, s.node_bits,
                                    w.rs_hist.as<uint32_t>(), w.rs_dtot.as<uint32_t>(), st, true);
    const uint32_t* su = in_tmp ? w.skey2.as<uint32_t>() : w.skey.as<uint32_t>();
    const uint32_t* se = in_tmp ? w.sval2.as<uint32_t>() : w.sval.as<uint32_t>();
    const int gH = (int)std::min<int64_t>(4096, std::max<int64_t>(1, (g.Smax + kHeadTile - 1) / kHeadTile));
    hipLaunchKernelGGL(k_heads, dim3(gH), dim3(kBlock), lds_h, st, g.H, w.req_off.as<int64_t>(),
                       w.e_off.as<int64_t>(), su, se, rlk, rlv, w.pk.as<int64_t>(), w.hl.as<int32_t>(), ctl);
    scan_counts64(w.pk.as<int64_t>(), w.pkx.as<int64_t>(), &ctl->S, g.Smax, &ctl->pktot, part, st);
    hipLaunchKernelGGL(k_runs, dim3(gS), dim3(kBlock), lds_h, st, g.H, w.req_off.as<int64_t>(),
                       w.e_off.as<int64_t>(), su, se, w.pk.as<int64_t>(), w.pkx.as<int64_t>(),
                       w.hl.as<int32_t>(), w.nl_key.as<uint64_t>(), w.nl_run.as<int32_t>(),
                       w.run_local.as<int32_t>(), ctl);
    hipLaunchKernelGGL(k_grp_hist, dim3(kGroupWGs), dim3(kBlock), (size_t)g.H * 4, st, w.nl_key.as<uint64_t>(),
                       g.H, w.ghist.as<int64_t>(), ctl);
    hipLaunchKernelGGL(k_grp_scan, dim3(g.H), dim3(kBlock), 0, st, w.ghist.as<int64_t>(), w.newcnt.as<int64_t>());
    hipLaunchKernelGGL(k_grp_rank, dim3(kGroupWGs), dim3(kBlock), (size_t)g.H * 8 + (size_t)kWavesPerBlock * g.H * 4,
                       st, w.nl_key.as<uint64_t>(),
                       w.nl_run.as<int32_t>(), g.H, g.jbits, w.ghist.as<int64_t>(), w.size.as<int32_t>(), g.capN,
                       w.nodes.as<int32_t>(), w.run_local.as<int32_t>(), w.nl_val.as<int32_t>(), ctl);
    hipLaunchKernelGGL(k_relabel, dim3(gS), dim3(kBlock), 0, st, w.pk.as<int64_t>(), w.pkx.as<int64_t>(), se,
                       w.run_local.as<int32_t>(), b.col[l].as<int32_t>(), ctl);
    const int gM = (int)std::min<int64_t>(4096, (g.rows_max + kMergeTile - 1) / kMergeTile);
    hipLaunchKernelGGL(k_merge, dim3(gM), dim3(kBlock), 0, st, rlk, rlv, w.nl_key.as<uint64_t>(),
                       w.nl_val.as<int32_t>(), w.rl_key[cur ^ 1].as<uint64_t>(), w.rl_val[cur ^ 1].as<int32_t>(),
                       ctl);
    AGNES_CHECK_HIP(hipGetLastError());
}

void begin_hyperbatch(const Store& s, Batch& b, const int32_t* targets, int32_t H, int32_t B,
                      const int32_t* fanouts, int32_t L, uint64_t seed, int64_t mb_base,
                      hipStream_t st) {
    AGNES_REQUIRE(b.state != kSampled, AGNES_ERR_INVALID, "the batch has a hyperbatch begun but not finished");
    // a batch still gathering: its buffers are in use until the gather ends
    if (b.state == kGathering) wait_batch(b);
    b.state = kIdle;
    Geometry g = plan(s, H, B, fanouts, L);
    SyncLayout y = sync_layout(H, L);
    Workspace& w = b.ws;
    reserve_workspace(w, g, y);
    if (!b.sampled) AGNES_CHECK_HIP(hipEventCreateWithFlags(&b.sampled, hipEventDisableTiming));
    if (!b.gathered) AGNES_CHECK_HIP(hipEventCreateWithFlags(&b.gathered, hipEventDisableTiming));
    b.store = &s;
    b.H = H; b.B = B; b.L = L;
    b.capN = g.capN;
    b.stream = st;
    for (int l = 0; l < L; l++) {
        b.row_ptr[l].reserve((size_t)(H * g.cap[l] + H) * 4);
        b.col[l].reserve((size_t)std::max<int64_t>(1, H * g.cap[l] * fanouts[l]) * 4);
    }
    Ctl* ctl = w.sync.as<Ctl>();
    int32_t* lsz = (int32_t*)((char*)w.sync.ptr + y.lsz);
    int64_t* ec = (int64_t*)((char*)w.sync.ptr + y.ecount);

    if (s.profile) AGNES_CHECK_HIP(hipEventRecord(w.ev[0], st));
    hipLaunchKernelGGL(k_ctl_init, dim3(1), dim3(kBlock), 0, st, ctl, (int64_t)H * B);
    hipLaunchKernelGGL(k_init, dim3(grid_for((int64_t)H * B, 1024)), dim3(kBlock), 0, st, targets, H, B,
                       s.num_nodes, g.capN, w.nodes.as<int32_t>(), w.size.as<int32_t>(), w.newcnt.as<int64_t>(),
                       w.skey.as<uint32_t>(), ctl);
    int in_tmp = radix_sort_pairs32(w.skey.as<uint32_t>(), w.sval.as<uint32_t>(), w.skey2.as<uint32_t>(),
                                    w.sval2.as<uint32_t>(), &ctl->targets, (int64_t)H * B, s.node_bits,
                                    w.rs_hist.as<uint32_t>(), w.rs_dtot.as<uint32_t>(), st, true);
    hipLaunchKernelGGL(k_list0, dim3(grid_for((int64_t)H * B, 1024)), dim3(kBlock), 0, st,
                       in_tmp ? w.skey2.as<uint32_t>() : w.skey.as<uint32_t>(),
                       in_tmp ? w.sval2.as<uint32_t>() : w.sval.as<uint32_t>(), B, w.rl_key[0].as<uint64_t>(),
                       w.rl_val[0].as<int32_t>(), ctl);
    AGNES_CHECK_HIP(hipGetLastError());
    int cur = 0;
    for (int l = 0; l < L; l++) {
        if (s.offsets64) launch_layer<int64_t>(s, w, g, l, fanouts[l], seed, mb_base, b, y, cur, st);
        else launch_layer<int32_t>(s, w, g, l, fanouts[l], seed, mb_base, b, y, cur, st);
        cur ^= 1;
    }
    b.cur = cur;
    // close the last hop: edge counts, final node counts, output row offsets
    hipLaunchKernelGGL(k_begin, dim3(1), dim3(kBlock), 0, st, L, L, H, ctl, w.size.as<int32_t>(),
                       w.newcnt.as<int64_t>(), lsz, ec, w.req_off.as<int64_t>(), w.e_off.as<int64_t>(),
                       w.mb_off.as<int64_t>());
    AGNES_CHECK_HIP(hipGetLastError());
    if (s.profile) AGNES_CHECK_HIP(hipEventRecord(w.ev[1], st));
    // sizes of the outputs travel to pinned host memory; finish reads them
    AGNES_CHECK_HIP(hipMemcpyAsync(w.sync_host.ptr, w.sync.ptr, y.bytes, hipMemcpyDeviceToHost, st));
    AGNES_CHECK_HIP(hipEventRecord(b.sampled, st));
    b.state = kSampled;
}

void finish_hyperbatch(Batch& b, hipStream_t st) {
    AGNES_REQUIRE(b.state == kSampled, AGNES_ERR_INVALID, "finish needs a begun hyperbatch");
    const Store& s = *b.store;
    Workspace& w = b.ws;
    const int H = b.H, L = b.L;
    SyncLayout y = sync_layout(H, L);
    AGNES_CHECK_HIP(hipEventSynchronize(b.sampled));
    b.state = kIdle;   // until the gather is enqueued
    Ctl hc;
    memcpy(&hc, w.sync_host.ptr, sizeof(Ctl));
    AGNES_REQUIRE(!(hc.err & 1), AGNES_ERR_INVALID, "a target is outside [0, num_nodes)");
    AGNES_REQUIRE(!(hc.err & 2), AGNES_ERR_INVALID, "a target appears twice in one minibatch");
    AGNES_REQUIRE(!(hc.err & 4), AGNES_ERR_INTERNAL, "node capacity exceeded");
    b.layer_sizes.assign((size_t)H * (L + 1), 0);
    memcpy(b.layer_sizes.data(), (char*)w.sync_host.ptr + y.lsz, b.layer_sizes.size() * 4);
    std::vector<int64_t> ecount((size_t)H * L);
    memcpy(ecount.data(), (char*)w.sync_host.ptr + y.ecount, ecount.size() * 8);
    memset(&b.stats, 0, sizeof(b.stats));
    b.stats.L = L;
    for (int l = 0; l < L; l++) {
        b.stats.requests[l] = hc.requests[l];
        b.stats.sampled[l] = hc.sampled[l];
        b.stats.new_nodes[l] = hc.new_nodes[l];
        b.stats.topo_blocks[l] = hc.topo_blocks[l];
    }

    // host view offsets
    b.node_off.assign((size_t)H + 1, 0);
    for (int j = 0; j < H; j++) b.node_off[j + 1] = b.node_off[j] + b.layer_sizes[(size_t)j * (L + 1) + L];
    for (int l = 0; l < L; l++) {
        b.rp_off[l].assign((size_t)H + 1, 0);
        b.col_off[l].assign((size_t)H + 1, 0);
        for (int j = 0; j < H; j++) {
            int64_t nd = b.layer_sizes[(size_t)j * (L + 1) + l];
            b.rp_off[l][j + 1] = b.rp_off[l][j] + nd + 1;
            int64_t ne = ecount[(size_t)j * L + l];
            AGNES_REQUIRE(ne < 0x7FFFFFFFll, AGNES_ERR_RANGE, "a minibatch has >= 2^31 edges in one hop");
            b.col_off[l][j + 1] = b.col_off[l][j] + ne;
        }
    }
    const int64_t rows = b.node_off[H];
    AGNES_REQUIRE(rows < 0x7FFFFFFFll, AGNES_ERR_RANGE, "more than 2^31-1 gathered rows");
    b.stats.rows = rows;
    b.nodes.reserve_slack((size_t)std::max<int64_t>(rows, 1) * 4);
    b.features.reserve_slack((size_t)std::max<int64_t>(rows, 1) * (size_t)s.row_bytes);

    // gather over the final list, ordered after the sampling phase
    if (st != b.stream) AGNES_CHECK_HIP(hipStreamWaitEvent(st, b.sampled, 0));
    Ctl* ctl = w.sync.as<Ctl>();
    if (s.profile) {
        AGNES_CHECK_HIP(hipEventRecord(w.ev[2], st));
        AGNES_CHECK_HIP(hipEventRecord(w.ev[3], st));
    }
    const uint64_t* rlk = w.rl_key[b.cur].as<uint64_t>();
    const int32_t* rlv = w.rl_val[b.cur].as<int32_t>();
    if (rows > 0) {
        if (s.row_bytes % 16 == 0)
            launch_gather<u32x4>(s.features.ptr, b.features.ptr, b.nodes.as<int32_t>(), rlk, rlv,
                                 w.mb_off.as<int64_t>(), H, rows, s.row_bytes / 16, (uint32_t)s.rpb, ctl,
                                 s.gather_groups, s.gather_unroll, st);
        else
            launch_gather<uint32_t>(s.features.ptr, b.features.ptr, b.nodes.as<int32_t>(), rlk, rlv,
                                    w.mb_off.as<int64_t>(), H, rows, s.row_bytes / 4, (uint32_t)s.rpb, ctl,
                                    s.gather_groups, s.gather_unroll, st);
    }
    AGNES_CHECK_HIP(hipGetLastError());
    if (s.profile) AGNES_CHECK_HIP(hipEventRecord(w.ev[4], st));
    AGNES_CHECK_HIP(hipMemcpyAsync(w.sync_host.ptr, ctl, sizeof(Ctl), hipMemcpyDeviceToHost, st));
    AGNES_CHECK_HIP(hipEventRecord(b.gathered, st));
    b.stream = st;
    b.state = kGathering;
}

void wait_batch(Batch& b) {
    if (b.state == kDone) return;
    AGNES_REQUIRE(b.state == kGathering, AGNES_ERR_INVALID, "the batch holds no finished hyperbatch");
    AGNES_CHECK_HIP(hipEventSynchronize(b.gathered));
    Ctl hc;
    memcpy(&hc, b.ws.sync_host.ptr, sizeof(Ctl));
    b.stats.distinct_rows = hc.distinct;
    b.stats.feat_blocks = hc.fblocks;
    b.stats.sample_ms = b.stats.gather_ms = b.stats.copy_ms = -1.0f;
    if (b.store->profile) {
        Workspace& w = b.ws;
        AGNES_CHECK_HIP(hipEventElapsedTime(&b.stats.sample_ms, w.ev[0], w.ev[1]));
        AGNES_CHECK_HIP(hipEventElapsedTime(&b.stats.gather_ms, w.ev[2], w.ev[4]));
        AGNES_CHECK_HIP(hipEventElapsedTime(&b.stats.copy_ms, w.ev[3], w.ev[4]));
    }
    b.state = kDone;
}

}  // namespace agnes
