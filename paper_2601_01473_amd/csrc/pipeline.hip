// The hyperbatch data-preparation pipeline (AGNES, arXiv 2601.01473, Alg. 1) on
// gfx950.
//
// The bucket matrix Bck of Sec. 3.4(3) (rows = blocks, columns = minibatches,
// cells = the nodes a minibatch needs from a block) is kept as one list of all
// (node, minibatch) pairs of the hyperbatch, sorted by node id and then by
// minibatch.  Objects are stored in ascending node order, so a block's row of
// Bck is a contiguous run of this list, and a node needed by several
// minibatches is a run inside it.  Each hop (Alg. 1, sampling loop):
//   counts      k = min(deg, f_l) per request, in (minibatch, row) order, with
//               the reduce pass of the edge-offset scan (k_count_reduce)
//   scan        edge offset of every request (the hop's row pointers)
//   k_sample    walks the list in block order: Floyd subsets from Philox words,
//               neighbours written at the request's edge offset
//   radix sort  the sampled neighbours by node id (stable: minibatch order kept)
//   join        merge path of the list with the sorted neighbours: a run of
//               equal (node, minibatch) keys is an old node when the list holds
//               the pair, else a new node; new nodes get local ids in id order
//               per minibatch, every edge gets its column, and the new pairs
//               are merged into the list (count, scan, write)
// Gather (Alg. 1, gathering loop): the final list is the feature bucket in block
// order; k_gather copies each row to every minibatch that needs it.
//
// Nothing here uses a device-wide atomic per element; every size stays on the
// device until one synchronisation before the gather.
#include <algorithm>
#include <cstring>
#include <functional>
#include <vector>

#include "bucket.hpp"
#include "device.hpp"
#include "runtime.hpp"

namespace agnes {

struct Geometry {
    int32_t H, B, L;
    int64_t capN;                      // node capacity of one minibatch
    int64_t cap[AGNES_MAX_LAYERS + 1]; // cap[l] = frontier capacity of hop l (cap[L] = capN)
    int64_t Rmax, Smax, rows_max, sort_max;
    int64_t ebound[AGNES_MAX_LAYERS];  // sampled edges of hop l at most: H cap[l] f_l
    int jbits;
    // node-range buckets: per hop the most coarse buckets and the count
    // table's row stride
    int bcoarse[AGNES_MAX_LAYERS], bstride[AGNES_MAX_LAYERS];
    int bstride_max;
};

// Edge numbers, sort positions and positions in the join of one hop are
// 32-bit: a hop whose requests plus sampled edges can reach 2^32 (bound
// H cap_l (1 + f_l)) is refused here, before anything is allocated or launched.
static Geometry plan(const Store& s, int32_t H, int32_t B, const int32_t* fanouts, int32_t L) {
    Geometry g{};
    g.H = H; g.B = B; g.L = L;
    g.cap[0] = B;
    g.Rmax = 0; g.Smax = 0;
    const int64_t nmax = std::max<int64_t>(s.num_nodes, B);
    for (int l = 0; l < L; l++) {
        const unsigned __int128 bound = (unsigned __int128)H * (uint64_t)g.cap[l] * (uint64_t)(1 + fanouts[l]);
        AGNES_REQUIRE(bound < ((unsigned __int128)1 << 32), AGNES_ERR_RANGE,
                      "a hop's requests and sampled edges can reach 2^32 (H * frontier capacity * (1 + fanout))");
        g.Rmax = std::max<int64_t>(g.Rmax, (int64_t)H * g.cap[l]);
        g.Smax = std::max<int64_t>(g.Smax, (int64_t)H * g.cap[l] * fanouts[l]);
        g.ebound[l] = (int64_t)H * g.cap[l] * fanouts[l];
        g.cap[l + 1] = std::min<int64_t>(g.cap[l] * (1 + (int64_t)fanouts[l]), nmax);
    }
    g.capN = g.cap[L];
    g.rows_max = (int64_t)H * g.capN;
    g.sort_max = std::max<int64_t>(g.Smax, (int64_t)H * B);
    int jb = 0;
    while ((1 << jb) < H) jb++;
    g.jbits = jb;
    g.bstride_max = kBlock;
    for (int l = 0; l < L; l++) {
        const int64_t load = (int64_t)H * g.cap[l] * (1 + (int64_t)fanouts[l]);
        const BucketBounds bb = bucket_bounds(s, load, H);
        g.bcoarse[l] = bb.coarse;
        g.bstride[l] = bucket_table_stride(bb);
        g.bstride_max = std::max(g.bstride_max, g.bstride[l]);
    }
    return g;
}

// Most workgroups of each looping sampling kernel (the sampler, the radix
// passes, the join) of a hop of at most `bound` sampled edges: the store's
// setting, or by default the power of two at or below bound / 32768, within
// [512, 2048].  Beside a running row copy fewer workgroups start sooner, while
// a large hop needs more to hide its latency; measured: 512 suits hops of
// about 2M edges (the 2^23-node workload), 2048 those of 15M (the 2^26-node
// workload's last hop).
static int hop_cap(const Store& s, int64_t bound) {
    if (s.sample_groups > 0) return s.sample_groups;
    int cap = 512;
    while (cap < 2048 && (int64_t)cap * 2 <= bound / 32768) cap *= 2;
    return cap;
}

// Workgroups of the sampler (k_sample) of hop l: a multiple of the XCD count.
static int hop_grid(const Store& s, const Geometry& g, int l) {
    const int G = grid_for((int64_t)g.H * g.cap[l], std::min(2048, hop_cap(s, g.ebound[l])));
    return (G + kXcds - 1) / kXcds * kXcds;
}

// ----------------------------------------------------------------- small kernels

__device__ __forceinline__ void load_offsets(int64_t* dst, const int64_t* src, int n) {
    for (int i = threadIdx.x; i <= n; i += kBlock) dst[i] = src[i];
    __syncthreads();
}

// Minibatch of edge e given the request offsets: mb_e[j] = e_off[req_off[j]].
__device__ __forceinline__ void load_mb_edges(int64_t* mb_e, const int64_t* req_off, const uint32_t* e_off, int H) {
    for (int i = threadIdx.x; i <= H; i += kBlock) mb_e[i] = (int64_t)e_off[req_off[i]];
    __syncthreads();
}

// Values that change from call to call.  The host hands them to k_params by
// value; every later kernel of the sampling phase reads them from device
// memory, so the same launches (or a graph captured from them) serve any call.
struct ChainParams {
    const int32_t* targets;   // [H][B] device
    uint64_t seed;
    int64_t mb_base;          // global index of minibatch 0
};

// Also clears the hyperbatch's counters (one launch instead of two at the head
// of every chain).
__global__ void k_params(ChainParams* p, const int32_t* targets, uint64_t seed, int64_t mb_base, Ctl* ctl,
                         int64_t ntargets) {
    int64_t* c = (int64_t*)ctl;
    for (int i = threadIdx.x; i < (int)(sizeof(Ctl) / 8); i += kBlock) c[i] = 0;
    __syncthreads();
    if (threadIdx.x == 0) {
        p->targets = targets;
        p->seed = seed;
        p->mb_base = mb_base;
        ctl->targets = ntargets;
    }
}

// Targets become the first B nodes of every minibatch.  An out-of-range target
// is recorded as an error and replaced by node 0 so that later kernels stay in
// bounds.  tkey receives the node ids for the sort that builds the list.
__global__ __launch_bounds__(kBlock) void k_init(const ChainParams* prm, int H, int B, int64_t num_nodes,
                                                 int64_t capN, int32_t* nodes, int32_t* size,
                                                 int64_t* newcnt, uint32_t* tkey, Ctl* ctl) {
    const int32_t* targets = prm->targets;
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
                                                  int64_t* req_off, const uint32_t* e_off, int64_t* node_off,
                                                  const uint32_t* topo_part, int n_part) {
    __shared__ int64_t lds[kWavesPerBlock];
    if (l > 0) {
        // the previous hop's non-empty Bck rows: the sampler's per-workgroup counts
        int64_t t = 0;
        for (int i = threadIdx.x; i < n_part; i += kBlock) t += topo_part[i];
        int64_t tot;
        (void)block_exclusive_scan(t, lds, tot);
        if (threadIdx.x == 0) ctl->topo_blocks[l - 1] = tot;
        for (int j = threadIdx.x; j < H; j += kBlock) {
            ecount[(int64_t)j * L + (l - 1)] = (int64_t)e_off[req_off[j + 1]] - (int64_t)e_off[req_off[j]];
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
    // after a node-range bucket overflowed (err bit 3) the hyperbatch is
    // sampled again on the radix-sort path: every later hop gets no requests
    const bool dead = (ctl->err & 8) != 0;
    int64_t carry = 0;
    for (int base = 0; base < H; base += kBlock) {
        int j = base + threadIdx.x;
        int64_t v = (j < H && !dead) ? size[j] : 0;
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

// Per-request counts fused with the reduce pass of the edge-offset scan: the counts of
// scan range g (scan_range over the hop's R requests, G ranges) and their sum
// in partials[g]; the scan's final pass follows.
template <typename OffT>
__global__ __launch_bounds__(kBlock) void k_count_reduce(int H, int64_t capN, int32_t f, const OffT* off,
                                                         const int32_t* nodes, const int64_t* req_off_g,
                                                         int32_t* cnt, int G, int64_t* partials, const Ctl* ctl) {
    extern __shared__ int64_t req_off[];
    __shared__ int64_t lds[kWavesPerBlock];
    load_offsets(req_off, req_off_g, H);
    int64_t lo, hi;
    scan_range(ctl->R, G, blockIdx.x, lo, hi);
    int64_t sum = 0;
    for (int64_t q = lo + threadIdx.x; q < hi; q += kBlock) {
        const int j = upper_segment(req_off, H, q);
        const int32_t v = nodes[(int64_t)j * capN + (q - req_off[j])];
        const int64_t deg = (int64_t)off[v + 1] - (int64_t)off[v];
        const int32_t k = (int32_t)(deg < f ? deg : f);
        cnt[q] = k;
        sum += k;
    }
    int64_t total;
    (void)block_exclusive_scan(sum, lds, total);
    if (threadIdx.x == 0) partials[blockIdx.x] = total;
}

// Sample every request of the hop, walking the list in (node, minibatch) order:
// consecutive threads serve the requests of the same topology block from every
// minibatch, and the requests of one node are neighbours.  Also counts the
// topology blocks the hop touches (non-empty rows of Bck).
template <typename OffT, int MAXK>
__global__ __launch_bounds__(kBlock) void k_sample(int l, int H, int32_t f, const ChainParams* prm,
                                                   const OffT* off, const int32_t* adj, int e_blk_log2,
                                                   int64_t nblk, const uint64_t* rl_key, const int32_t* rl_val,
                                                   const int64_t* req_off_g, const uint32_t* e_off,
                                                   int32_t* cg, uint32_t* topo_part, const Ctl* ctl) {
    extern __shared__ int64_t req_off[];      // [H+1] request offsets
    __shared__ uint32_t opened;
    const uint64_t seed = prm->seed;
    const int64_t mb_base = prm->mb_base;
    if (threadIdx.x == 0) opened = 0;
    load_offsets(req_off, req_off_g, H);
    const int64_t R = ctl->R;
    // XCD x (workgroups dealt to the 8 XCDs in turn; the grid is a multiple of
    // 8) walks the x-th eighth of the list, so the lines that neighbouring
    // requests share (offsets, edge offsets of a minibatch's consecutive rows)
    // are fetched into one L2 rather than eight
    const int xcd = (int)(blockIdx.x % kXcds);
    const int64_t part = ((R + kXcds - 1) / kXcds + kBlock - 1) / kBlock * kBlock;
    const int64_t lo = std::min<int64_t>(R, (int64_t)xcd * part), hi = std::min<int64_t>(R, lo + part);
    const int64_t stride = (int64_t)(gridDim.x / kXcds) * kBlock;
    const int64_t first = lo + (int64_t)(blockIdx.x / kXcds) * kBlock;
    // the next request's list entry is loaded while this one is sampled
    uint64_t next_key = 0;
    int32_t next_val = 0;
    {
        const int64_t p0 = first + threadIdx.x;
        if (p0 < hi) {
            next_key = rl_key[p0];
            next_val = rl_val[p0];
        }
    }
    for (int64_t base = first; base < hi; base += stride) {
        int64_t p = base + threadIdx.x;
        bool active = p < hi;
        int64_t blk = -1;
        const uint64_t key = next_key;
        const int32_t val = next_val;
        if (p + stride < hi) {
            next_key = rl_key[p + stride];
            next_val = rl_val[p + stride];
        }
        if (active) {
            int32_t v = (int32_t)(key >> 32);
            int j = (int)(uint32_t)key;
            int64_t r = val;
            int64_t q = req_off[j] + r;
            int64_t o0 = (int64_t)off[v];
            int64_t deg = (int64_t)off[v + 1] - o0;
            blk = o0 >> e_blk_log2;
            if (blk >= nblk) blk = nblk - 1;
            int k = (int)(deg < f ? deg : f);
            int64_t eo = (int64_t)e_off[q];
            int32_t* out = cg + eo;
            const int32_t* a = adj + o0;
            if (MAXK > 0) {
                // positions (all of them for a take-all row), then one round of loads
                constexpr int MK = MAXK > 0 ? MAXK : 1;
                uint32_t pos[MK];
                if (k == deg) {
#pragma unroll
                    for (int i = 0; i < MK; i++) pos[i] = (uint32_t)i;
                } else {
                    floyd_positions<MK>((uint64_t)deg, k, seed, (uint64_t)v, (uint64_t)(mb_base + j),
                                        (uint64_t)l, pos);
                }
                write_ranked<MK>(pos, k, a, out);
            } else if (k == deg) {
                copy_row(a, k, out);
            } else {
                floyd_sample_mem((uint64_t)deg, k, seed, (uint64_t)v, (uint64_t)(mb_base + j), (uint64_t)l, a, out);
            }
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
        if (lane_id() == 0 && m) atomicAdd(&opened, (uint32_t)__popcll(m));
    }
    // one count per workgroup (summed by the next k_begin): a device-wide
    // atomic per wave on one address would serialize
    __syncthreads();
    if (threadIdx.x == 0) topo_part[blockIdx.x] = opened;
}

// ----------------------------------------------------------------- join
//
// After the sort, the hop's sampled edges B (keys (node, minibatch), sorted,
// equal keys in edge order) are joined with the list A of the pairs already
// held (sorted, unique keys, value = local id).  Both are ordered by key with A
// first on equal keys, so the pair of a run of equal edge keys, if A holds it,
// sits right before the run.  Merge path cuts the merged sequence into tiles of
// kJoinTile entries: tile t holds A[a_t, a_{t+1}) and B[t*T - a_t, ...) with
// a_t from k_join_count.  An edge whose key differs from the previous edge's
// is a run head; a head whose pair A holds is an old node (the pair is in the
// tile's A part or is A[a_t - 1]), otherwise a new one.  New nodes take local
// ids |S_{j,l-1}| + (rank among the new nodes of minibatch j in key order), so
// each minibatch's new nodes are ascending by id.  G workgroups take
// consecutive runs of tiles: k_join_count counts the new nodes per minibatch
// and the merged-list entries of every group, k_join_scan turns the counts into
// offsets, k_join_write emits the merged list (A's entries and one entry per
// new pair, in key order), the new nodes' ids and every edge's column.  The
// number of groups G is a multiple of 256 chosen by the host (join_groups).
constexpr int kJoinTile = 1024;                               // merged entries per tile
constexpr int kJoinWaveItems = kJoinTile / kWavesPerBlock;    // edges of a tile per wave
constexpr int kJoinRounds = kJoinWaveItems / kWave;
constexpr uint64_t kNoKey = ~0ull;                            // no pair has this key (node < 2^31)

__device__ __forceinline__ uint64_t edge_key(const uint32_t* su, const uint32_t* se, const int64_t* mb_e, int H,
                                             int64_t p) {
    return ((uint64_t)su[p] << 32) | (uint32_t)upper_segment(mb_e, H, (int64_t)se[p]);
}

// Merge path: a_t, the number of A entries among the first t * kJoinTile
// merged entries, is found for every tile boundary t by groups of
// kSplitLanes lanes (a few rounds of 16 probes) in k_join_count.
constexpr int kSplitLanes = 16;

struct JoinSpan {
    int64_t a0, b0;
    int nA, nB;
};

__device__ __forceinline__ JoinSpan join_span(int64_t t, int64_t n, const int64_t* split) {
    JoinSpan s;
    const int64_t d0 = t * kJoinTile, d1 = std::min<int64_t>(d0 + kJoinTile, n);
    s.a0 = split[0];
    const int64_t a1 = split[1];
    s.b0 = d0 - s.a0;
    s.nA = (int)(a1 - s.a0);
    s.nB = (int)((d1 - a1) - s.b0);
    return s;
}

// A tile's entries, one thread's share in registers: merged slot
// m = tid + k kBlock (k < kJoinSlots) is A[a0 + m] for m < nA (key, local id)
// and edge b0 + m - nA for nA <= m < nA + nB (node, edge number).  Thread 0
// also holds the entries just before the tile.  The loads for tile t + 1 are
// issued before tile t is processed, so their latency hides behind that work
// (a workgroup barrier waits for LDS operations only).
constexpr int kJoinSlots = kJoinTile / kBlock;
static_assert(kJoinTile % kBlock == 0, "whole slots per thread");

struct JoinRegs {
    uint64_t k[kJoinSlots];
    int32_t v[kJoinSlots];
    uint64_t pk;         // thread 0: A[a0 - 1] (kNoKey if none)
    int32_t pv;          // its local id
    uint32_t pu, pe;     // thread 0: node and edge number of edge b0 - 1 (if b0 > 0)
};

__device__ __forceinline__ void join_load(const JoinSpan& s, const uint64_t* ak, const int32_t* av,
                                          const uint32_t* su, const uint32_t* se, JoinRegs& r) {
#pragma unroll
    for (int k = 0; k < kJoinSlots; k++) {
        const int m = threadIdx.x + k * kBlock;
        if (m < s.nA) {
            r.k[k] = ak[s.a0 + m];
            r.v[k] = av[s.a0 + m];
        } else if (m < s.nA + s.nB) {
            const int64_t p = s.b0 + (m - s.nA);
            r.k[k] = su[p];
            r.v[k] = (int32_t)se[p];
        }
    }
    if (threadIdx.x == 0) {
        r.pk = s.a0 > 0 ? ak[s.a0 - 1] : kNoKey;
        r.pv = s.a0 > 0 ? av[s.a0 - 1] : 0;
        r.pu = s.b0 > 0 ? su[s.b0 - 1] : 0u;
        r.pe = s.b0 > 0 ? se[s.b0 - 1] : 0u;
    }
}

// The tile in LDS: sk[0, nA) = A keys, sk[nA, nA + nB) = edge keys (node,
// minibatch); sv = A local ids, then edge numbers.  pre = {key of the edge
// before the tile, key of the A entry before the tile} (kNoKey if none),
// pre_val = that A entry's local id.
__device__ __forceinline__ void join_store(const JoinSpan& s, const JoinRegs& r, const int64_t* mb_e, int H,
                                           uint64_t* sk, int32_t* sv, uint64_t* pre, int32_t* pre_val) {
#pragma unroll
    for (int k = 0; k < kJoinSlots; k++) {
        const int m = threadIdx.x + k * kBlock;
        if (m < s.nA) {
            sk[m] = r.k[k];
            sv[m] = r.v[k];
        } else if (m < s.nA + s.nB) {
            const uint32_t e = (uint32_t)r.v[k];
            sk[m] = (r.k[k] << 32) | (uint32_t)upper_segment(mb_e, H, (int64_t)e);
            sv[m] = r.v[k];
        }
    }
    if (threadIdx.x == 0) {
        pre[0] = s.b0 > 0 ? (((uint64_t)r.pu << 32) | (uint32_t)upper_segment(mb_e, H, (int64_t)r.pe)) : kNoKey;
        pre[1] = r.pk;
        *pre_val = r.pv;
    }
}

// Edge i of the tile (key K): head?  For a head, idx = lower bound of K in the
// tile's A part, and found / floc = whether A holds K and its local id.
struct EdgeFlags {
    bool head, found;
    int idx;
    int32_t floc;
};

// Lower bounds of Q keys in the sorted sk[lo, hi), searched in lockstep: a
// fixed sequence of halving steps, the same for every key and lane, so the Q
// searches' LDS reads overlap.  The answer stays in [base, base + n].
template <int Q>
__device__ __forceinline__ void lds_lower_bounds(const uint64_t* sk, int lo, int hi, const uint64_t (&key)[Q],
                                                 int (&out)[Q]) {
    int base[Q];
#pragma unroll
    for (int q = 0; q < Q; q++) base[q] = lo;
    int n = hi - lo;
    while (n > 1) {
        const int half = n >> 1;
#pragma unroll
        for (int q = 0; q < Q; q++) base[q] = sk[base[q] + half] < key[q] ? base[q] + half : base[q];
        n -= half;
    }
#pragma unroll
    for (int q = 0; q < Q; q++) out[q] = (n == 1 && sk[base[q]] < key[q]) ? base[q] + 1 : base[q];
}

// Edges i[q] of the tile (valid[q]: i[q] < nB): their keys, whether each is a
// head and, for a head, idx = lower bound of its key in the tile's A part and
// found / floc = whether A holds the key and its local id.  The Q searches run
// together (lds_lower_bounds).
template <int Q>
__device__ __forceinline__ void edge_flags(const uint64_t* sk, const int32_t* sv, int nA, const int (&i)[Q],
                                           const bool (&valid)[Q], uint64_t (&K)[Q], const uint64_t* pre,
                                           int32_t pre_val, EdgeFlags (&f)[Q]) {
#pragma unroll
    for (int q = 0; q < Q; q++) {
        K[q] = valid[q] ? sk[nA + i[q]] : 0;
        const uint64_t prevK = (valid[q] && i[q] > 0) ? sk[nA + i[q] - 1] : pre[0];
        f[q] = EdgeFlags{valid[q] && K[q] != prevK, false, 0, 0};
    }
    int lb[Q];
    lds_lower_bounds<Q>(sk, 0, nA, K, lb);
#pragma unroll
    for (int q = 0; q < Q; q++) {
        if (!f[q].head) continue;
        f[q].idx = lb[q];
        if (lb[q] < nA && sk[lb[q]] == K[q]) {
            f[q].found = true;
            f[q].floc = sv[lb[q]];
        } else if (pre[1] == K[q]) {
            f[q].found = true;
            f[q].floc = pre_val;
        }
    }
}

__device__ __forceinline__ void group_tiles(int64_t n, int g, int G, int64_t& t0, int64_t& t1) {
    const int64_t tiles = (n + kJoinTile - 1) / kJoinTile;
    const int64_t per = (tiles + G - 1) / G;
    t0 = std::min<int64_t>(tiles, (int64_t)g * per);
    t1 = std::min<int64_t>(tiles, t0 + per);
}

// Pass 1: per group, the merge-path boundaries of its tiles (into split, for
// pass 2 too: a_t of every tile boundary t, searched by groups of kSplitLanes
// lanes), new nodes per minibatch (ghist[j][g]) and merged entries
// (gemit[g]).  Also writes the hop's row pointers in request order: row r of
// minibatch j starts at its edge offset minus the minibatch's first edge.
// Dynamic LDS: mb_e[H+1], ro[H+1], sk[T], sv[T], count[H], ssplit[per].
__global__ __launch_bounds__(kBlock) void k_join_count(int H, const int64_t* req_off, const uint32_t* e_off,
                                                       const uint64_t* ak, const int32_t* av, const uint32_t* su,
                                                       const uint32_t* se, int64_t* split, int G,
                                                       int64_t* ghist, int64_t* gemit, int32_t* row_ptr,
                                                       const Ctl* ctl) {
    extern __shared__ int64_t lds[];
    int64_t* mb_e = lds;
    int64_t* ro = mb_e + H + 1;
    uint64_t* sk = (uint64_t*)(ro + H + 1);
    int32_t* sv = (int32_t*)(sk + kJoinTile);
    uint32_t* count = (uint32_t*)(sv + kJoinTile);
    int64_t* ssplit = (int64_t*)(((uintptr_t)(count + H) + 7) & ~(uintptr_t)7);
    __shared__ uint64_t pre[2];
    __shared__ int32_t pre_val;
    __shared__ uint32_t nh_total;
    const int tid = threadIdx.x, g = blockIdx.x;
    for (int j = tid; j < H; j += kBlock) count[j] = 0;
    if (tid == 0) nh_total = 0;
    for (int i = tid; i <= H; i += kBlock) ro[i] = req_off[i];
    load_mb_edges(mb_e, req_off, e_off, H);
    const int64_t R = ctl->R;
    for (int64_t q = (int64_t)g * kBlock + tid; q < R; q += (int64_t)G * kBlock) {
        const int j = upper_segment(ro, H, q);
        row_ptr[q + j] = (int32_t)((int64_t)e_off[q] - mb_e[j]);
        if (q + 1 == ro[j + 1]) row_ptr[q + j + 1] = (int32_t)((int64_t)e_off[q + 1] - mb_e[j]);
    }
    const int64_t nb = ctl->S, n = R + nb;
    int64_t t0, t1;
    group_tiles(n, g, G, t0, t1);
    // boundaries t0 .. t1: A[i] goes before B[d-1-i] when A[i] <= B[d-1-i]
    // (A first on equal keys); a neighbouring group writes the same value at
    // a shared boundary
    for (int64_t t = t0 + tid / kSplitLanes; t <= t1; t += kBlock / kSplitLanes) {
        const int64_t d = std::min<int64_t>(t * kJoinTile, n);
        const int64_t lo = d > nb ? d - nb : 0, hi = d < R ? d : R;
        const int64_t x = group_partition_point<kSplitLanes>(
            lo, hi, [&](int64_t i) { return ak[i] <= edge_key(su, se, mb_e, H, d - 1 - i); });
        if (lane_id() % kSplitLanes == 0) {
            ssplit[t - t0] = x;
            split[t] = x;
        }
    }
    __syncthreads();
    int64_t a_total = 0;
    uint32_t nh = 0;
    JoinRegs regs;
    if (t0 < t1) join_load(join_span(t0, n, ssplit), ak, av, su, se, regs);
    for (int64_t t = t0; t < t1; t++) {
        const JoinSpan s = join_span(t, n, ssplit + (t - t0));
        join_store(s, regs, mb_e, H, sk, sv, pre, &pre_val);
        if (t + 1 < t1) join_load(join_span(t + 1, n, ssplit + (t + 1 - t0)), ak, av, su, se, regs);
        a_total += s.nA;
        __syncthreads();
        {
            int ii[kJoinSlots];
            bool vv[kJoinSlots];
            uint64_t K[kJoinSlots];
            EdgeFlags f[kJoinSlots];
#pragma unroll
            for (int k = 0; k < kJoinSlots; k++) {
                ii[k] = tid + k * kBlock;
                vv[k] = ii[k] < s.nB;
            }
            edge_flags<kJoinSlots>(sk, sv, s.nA, ii, vv, K, pre, pre_val, f);
#pragma unroll
            for (int k = 0; k < kJoinSlots; k++) {
                if (f[k].head && !f[k].found) {
                    atomicAdd(&count[(uint32_t)K[k]], 1u);
                    nh++;
                }
            }
        }
        __syncthreads();
    }
    if (nh) atomicAdd(&nh_total, nh);
    __syncthreads();
    for (int j = tid; j < H; j += kBlock) ghist[(int64_t)j * G + g] = count[j];
    if (tid == 0) gemit[g] = a_total + nh_total;
}

// Workgroup j < H: exclusive scan of minibatch j's counts over the groups and
// its new-node total; workgroup H: the same for the merged entries, and the
// hop's new-node total (merged entries minus the old list).
__global__ __launch_bounds__(kBlock) void k_join_scan(int H, int G, int64_t* ghist, int64_t* gemit,
                                                      int64_t* newcnt, Ctl* ctl) {
    __shared__ int64_t lds[kWavesPerBlock];
    const int x = blockIdx.x;
    int64_t* row = x < H ? ghist + (int64_t)x * G : gemit;
    const int per = G / kBlock;                // G is a multiple of kBlock
    int64_t* mine = row + (int64_t)threadIdx.x * per;
    int64_t local = 0;
    for (int k = 0; k < per; k++) local += mine[k];
    int64_t total;
    int64_t ex = block_exclusive_scan(local, lds, total);
    for (int k = 0; k < per; k++) {
        const int64_t v = mine[k];
        mine[k] = ex;
        ex += v;
    }
    if (threadIdx.x == 0) {
        if (x < H) newcnt[x] = total;
        else ctl->n_new = total - ctl->R;
    }
}

// Pass 2.  Wave w takes a quarter of the tile's edges in rounds of 64;
// ballots give each edge the new heads before it in the wave and, for a new
// head, its rank among the wave's new heads of the same minibatch (wave-private
// counts wcnt[w][j]); after a barrier the waves' totals are stacked.  An edge
// takes the local id of the last head at or before it (a head before the tile:
// the old pair A[a_t - 1], or the newest new node of its minibatch so far).
// New nodes go to nodes (the per-minibatch lists: the next hop's requests, and
// after the last hop the output lists that k_list_stats packs).
// Dynamic LDS: mb_e[H+1], sk[T], sv[T], loc[T], nhx[T+1], cursor[H], wcnt[4][H] (16-bit),
// ssplit[per] (the group's tile boundaries).
__global__ __launch_bounds__(kBlock) void k_join_write(int H, int jbits, int64_t capN, int64_t rows_cap,
                                                       const int64_t* req_off, const uint32_t* e_off,
                                                       const uint64_t* ak, const int32_t* av, const uint32_t* su,
                                                       const uint32_t* se, const int64_t* split, int G,
                                                       const int64_t* ghist, const int64_t* gemit,
                                                       const int32_t* size, int32_t* nodes, uint64_t* ck,
                                                       int32_t* cv, int32_t* col, Ctl* ctl) {
    extern __shared__ int64_t lds[];
    int64_t* mb_e = lds;
    uint64_t* sk = (uint64_t*)(mb_e + H + 1);
    int32_t* sv = (int32_t*)(sk + kJoinTile);
    int32_t* loc = sv + kJoinTile;
    int32_t* nhx = loc + kJoinTile;
    int32_t* cursor = nhx + kJoinTile + 1;
    uint16_t* wcnt = (uint16_t*)(cursor + H);
    int64_t* ssplit = (int64_t*)(((uintptr_t)(wcnt + kWavesPerBlock * H) + 7) & ~(uintptr_t)7);
    __shared__ uint64_t pre[2];
    __shared__ int32_t pre_val, cont_local;
    __shared__ int32_t wnh[kWavesPerBlock], wanc[kWavesPerBlock];
    const int tid = threadIdx.x, w = wave_id(), lane = lane_id(), g = blockIdx.x;
    for (int j = tid; j < H; j += kBlock) {
        cursor[j] = size[j] + (int32_t)ghist[(int64_t)j * G + g];
        for (int x = 0; x < kWavesPerBlock; x++) wcnt[x * H + j] = 0;
    }
    const int64_t n = ctl->R + ctl->S;
    int64_t t0, t1;
    group_tiles(n, g, G, t0, t1);
    for (int64_t t = t0 + tid; t <= t1; t += kBlock) ssplit[t - t0] = split[t];
    load_mb_edges(mb_e, req_off, e_off, H);  // ends with a barrier
    int64_t run = gemit[g];                  // merged entries before the tile
    const uint64_t lane_le = lanemask_lt() | (1ull << lane);
    JoinRegs regs;
    if (t0 < t1) join_load(join_span(t0, n, ssplit), ak, av, su, se, regs);
    for (int64_t t = t0; t < t1; t++) {
        const JoinSpan s = join_span(t, n, ssplit + (t - t0));
        join_store(s, regs, mb_e, H, sk, sv, pre, &pre_val);
        if (t + 1 < t1) join_load(join_span(t + 1, n, ssplit + (t + 1 - t0)), ak, av, su, se, regs);
        __syncthreads();
        if (tid == 0) {
            // edges at the start of the tile that continue a run begun before it
            int32_t c = 0;
            if (s.nB > 0 && sk[s.nA] == pre[0]) c = (pre[1] == pre[0]) ? pre_val : cursor[(uint32_t)pre[0]] - 1;
            cont_local = c;
        }
        uint64_t key[kJoinRounds];
        int32_t nhw[kJoinRounds], jrk[kJoinRounds], anc[kJoinRounds], idx[kJoinRounds], floc[kJoinRounds];
        uint32_t kind = 0;                   // per round: bit 2r = head, bit 2r+1 = new
        int nh_run = 0, anc_run = -1;
        int items[kJoinRounds];
        bool inb[kJoinRounds];
        EdgeFlags fl[kJoinRounds];
#pragma unroll
        for (int r = 0; r < kJoinRounds; r++) {
            items[r] = w * kJoinWaveItems + r * kWave + lane;
            inb[r] = items[r] < s.nB;
        }
        edge_flags<kJoinRounds>(sk, sv, s.nA, items, inb, key, pre, pre_val, fl);
#pragma unroll
        for (int r = 0; r < kJoinRounds; r++) {
            const uint64_t K = key[r];
            const EdgeFlags f = fl[r];
            const bool nh = f.head && !f.found;
            const uint64_t nhm = __ballot(nh);
            nhw[r] = nh_run + __popcll(nhm & lanemask_lt());
            nh_run += __popcll(nhm);
            // rank among this wave's new heads of the same minibatch (lane order, then round order)
            const int j = (int)(uint32_t)K;
            uint64_t peers = nhm;
            for (int bit = 0; bit < jbits; bit++) {
                const uint64_t m = __ballot((j >> bit) & 1);
                peers &= ((j >> bit) & 1) ? m : ~m;
            }
            const int rank = __popcll(peers & lanemask_lt());
            const int leader = nh ? (__ffsll((unsigned long long)peers) - 1) : lane;
            int old = 0;
            if (nh && rank == 0) {
                old = wcnt[w * H + j];
                wcnt[w * H + j] = (uint16_t)(old + __popcll(peers));
            }
            old = __shfl(old, leader, kWave);
            jrk[r] = old + rank;
            // last head at or before this edge in the wave
            const uint64_t hm = __ballot(f.head);
            const uint64_t le = hm & lane_le;
            const int base = w * kJoinWaveItems + r * kWave;
            anc[r] = le ? base + 63 - __clzll(le) : anc_run;
            if (hm) anc_run = base + 63 - __clzll(hm);
            idx[r] = f.idx;
            floc[r] = f.floc;
            kind |= ((f.head ? 1u : 0u) | (nh ? 2u : 0u)) << (2 * r);
        }
        if (lane == 0) {
            wnh[w] = nh_run;
            wanc[w] = anc_run;
        }
        __syncthreads();
        int nh_base = 0, nh_total = 0, anc_carry = -1;
#pragma unroll
        for (int x = 0; x < kWavesPerBlock; x++) {
            if (x < w) {
                nh_base += wnh[x];
                anc_carry = std::max(anc_carry, wanc[x]);
            }
            nh_total += wnh[x];
        }
#pragma unroll
        for (int r = 0; r < kJoinRounds; r++) {
            const int i = w * kJoinWaveItems + r * kWave + lane;
            if (i >= s.nB) continue;
            nhx[i] = nh_base + nhw[r];
            if (anc[r] < 0) anc[r] = anc_carry;
            if ((kind >> (2 * r)) & 1u) {
                int32_t lc = floc[r];
                if ((kind >> (2 * r)) & 2u) {
                    const int j = (int)(uint32_t)key[r];
                    int rank = jrk[r];
                    for (int x = 0; x < w; x++) rank += wcnt[x * H + j];
                    lc = cursor[j] + rank;
                    const int64_t pos = run + idx[r] + nh_base + nhw[r];
                    if (lc >= capN || pos >= rows_cap) {
                        atomicOr((unsigned long long*)&ctl->err, 4ull);
                    } else {
                        nodes[(int64_t)j * capN + lc] = (int32_t)(key[r] >> 32);
                        ck[pos] = key[r];
                        cv[pos] = lc;
                    }
                }
                loc[i] = lc;
            }
        }
        if (tid == 0) nhx[s.nB] = nh_total;
        __syncthreads();
        // every edge's column; A's entries at their merged positions
#pragma unroll
        for (int r = 0; r < kJoinRounds; r++) {
            const int i = w * kJoinWaveItems + r * kWave + lane;
            if (i < s.nB) col[sv[s.nA + i]] = anc[r] >= 0 ? loc[anc[r]] : cont_local;
        }
        {
            uint64_t AK[kJoinSlots];
            int lb[kJoinSlots];
#pragma unroll
            for (int k = 0; k < kJoinSlots; k++) {
                const int ia = tid + k * kBlock;
                AK[k] = ia < s.nA ? sk[ia] : 0;
            }
            lds_lower_bounds<kJoinSlots>(sk, s.nA, s.nA + s.nB, AK, lb);
#pragma unroll
            for (int k = 0; k < kJoinSlots; k++) {
                const int ia = tid + k * kBlock;
                if (ia >= s.nA) continue;
                const int64_t pos = run + ia + nhx[lb[k] - s.nA];
                if (pos < rows_cap) {
                    ck[pos] = AK[k];
                    cv[pos] = sv[ia];
                }
            }
        }
        for (int j = tid; j < H; j += kBlock) {
            int tot = 0;
            for (int x = 0; x < kWavesPerBlock; x++) {
                tot += wcnt[x * H + j];
                wcnt[x * H + j] = 0;
            }
            cursor[j] += tot;
        }
        run += s.nA + nh_total;
        __syncthreads();
    }
}

// Tiles of the join at any hop: the list and the edges together fit the maxima.
static int64_t join_tiles_max(const Geometry& g) { return (g.Rmax + g.Smax) / kJoinTile + 1; }

// A group of the join passes keeps the merge-path boundaries of its tiles in
// LDS, so it takes at most this many tiles.
constexpr int64_t kJoinGroupTilesMax = 2048;

// Fewest groups that keep every group within kJoinGroupTilesMax tiles.
static int64_t join_groups_min(int64_t tiles) {
    const int64_t G = (tiles + kJoinGroupTilesMax - 1) / kJoinGroupTilesMax;
    return (G + kBlock - 1) / kBlock * kBlock;
}

// Workgroups of the join passes: one tile each up to 4096 groups, while the
// per-minibatch count table (H x G) stays near 4M entries; never fewer than
// join_groups_min.  A multiple of kBlock.
static int join_groups(int H, int64_t tiles) {
    int64_t G = std::min<int64_t>(4096, std::max<int64_t>(256, (int64_t)(4 << 20) / H));
    G = std::min<int64_t>(G, std::max<int64_t>(256, tiles));
    G = (G + kBlock - 1) / kBlock * kBlock;
    return (int)std::max<int64_t>(G, join_groups_min(tiles));
}

// per: the most tile boundaries of one group (its tiles + 1), at most
// kJoinGroupTilesMax + 2
static size_t join_count_lds(int H, int64_t per) {
    return (size_t)(H + 1) * 16 + (size_t)kJoinTile * 12 + (size_t)H * 4 + 8 + (size_t)per * 8;
}
static size_t join_write_lds(int H, int64_t per) {
    return (size_t)(H + 1) * 8 + (size_t)kJoinTile * 8 + (size_t)kJoinTile * 4 * 3 + 4 + (size_t)H * 4 +
           (size_t)kWavesPerBlock * H * 2 + 8 + (size_t)per * 8;
}

// Statistics of the final list (the feature bucket): distinct rows (runs of one
// node) and non-empty feature-block rows (runs of one feature block), one
// partial pair per workgroup for the host to add up.  With nodes_out, also the
// output node lists: minibatch j's list (nodes_ws[j capN ..], local-id order)
// is packed to nodes_out[node_off[j] ..], read and written in consecutive
// order (the row copy, which meets the entries in node order, would store each
// id alone at a scattered place).  Runs on the sampling stream so that the row
// copy does nothing but copy.
constexpr int kStatItems = 8;   // entries per thread per round (independent loads in flight)

__global__ __launch_bounds__(kBlock) void k_list_stats(const uint64_t* rl_key, uint32_t rpb, uint64_t* part,
                                                       const Ctl* ctl, const int32_t* nodes_ws, int64_t capN,
                                                       const int64_t* node_off_g, int H, int32_t* nodes_out) {
    extern __shared__ int64_t node_off[];      // [H+1] when nodes_out is given
    __shared__ unsigned long long cnt[2];
    if (threadIdx.x < 2) cnt[threadIdx.x] = 0;
    __syncthreads();
    const int64_t n = ctl->rows;
    // (not after a node-capacity error: the sizes may then exceed capN)
    // kStatItems entries per thread per round, all loaded before any is stored
    if (nodes_out && !(ctl->err & 4)) {
        load_offsets(node_off, node_off_g, H);
        const int64_t stride = (int64_t)gridDim.x * kBlock;
        for (int64_t b = (int64_t)blockIdx.x * kBlock + threadIdx.x; b < n; b += stride * kStatItems) {
            int64_t x[kStatItems];
            int j[kStatItems];
            int32_t v[kStatItems];
#pragma unroll
            for (int k = 0; k < kStatItems; k++) x[k] = std::min<int64_t>(b + k * stride, n - 1);
            upper_segments<kStatItems>(node_off, H, x, j);
#pragma unroll
            for (int k = 0; k < kStatItems; k++) v[k] = nodes_ws[(int64_t)j[k] * capN + (x[k] - node_off[j[k]])];
#pragma unroll
            for (int k = 0; k < kStatItems; k++)
                if (b + k * stride < n) nodes_out[b + k * stride] = v[k];
        }
    }
    unsigned long long nd = 0, nf = 0;
    const int64_t step = (int64_t)gridDim.x * kBlock * kStatItems;
    for (int64_t b = (int64_t)blockIdx.x * kBlock * kStatItems + threadIdx.x; b < n; b += step) {
        uint32_t u[kStatItems], pu[kStatItems];
#pragma unroll
        for (int i = 0; i < kStatItems; i++) {
            const int64_t e = b + (int64_t)i * kBlock;
            u[i] = e < n ? (uint32_t)(rl_key[e] >> 32) : 0u;
            pu[i] = (e > 0 && e < n) ? (uint32_t)(rl_key[e - 1] >> 32) : 0xFFFFFFFFu;
        }
#pragma unroll
        for (int i = 0; i < kStatItems; i++) {
            if (b + (int64_t)i * kBlock >= n) continue;
            nd += (pu[i] != u[i]);
            nf += (pu[i] == 0xFFFFFFFFu || pu[i] / rpb != u[i] / rpb);
        }
    }
    nd = wave_inclusive_scan(nd);
    nf = wave_inclusive_scan(nf);
    if (lane_id() == kWave - 1) {
        if (nd) atomicAdd(&cnt[0], nd);
        if (nf) atomicAdd(&cnt[1], nf);
    }
    __syncthreads();
    // one pair per workgroup, summed on the host (no device-wide atomics)
    if (threadIdx.x == 0) {
        part[2 * blockIdx.x] = cnt[0];
        part[2 * blockIdx.x + 1] = cnt[1];
    }
}

// ----------------------------------------------------------------- gather

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Source row of node u in the staged tier: its feature-cache row when it has
// one (the cache rows follow the pool's), else row (u mod rpb) of the pool
// slot that holds u's feature block.
__device__ __forceinline__ uint32_t source_row(const int32_t* tbuf, uint32_t rpb, const int32_t* tch,
                                               uint32_t pool_rows, uint32_t u) {
    if (tch) {
        const int32_t c = tch[u];
        if (c >= 0) return pool_rows + (uint32_t)c;
    }
    const uint32_t b = u / rpb;
    return (uint32_t)tbuf[b] * rpb + (u - b * rpb);
}

// Row copy over the final list, which is the feature bucket of Alg. 1's
// gathering loop in block order: the requests of a feature block are contiguous
// and those of one node are neighbours, so each row is loaded from HBM once and
// written to every minibatch that needs it (dest = node_off[j] + local id).
// LPR lanes share a row (16-byte or 4-byte units).  Lane groups take blocks of
// U consecutive entries in grid-stride order, so the waves in flight work on
// one compact window of the list: a minibatch's rows are written in ascending
// address order (the list is sorted by node, and so are the local ids of each
// hop's new nodes), and a compact window keeps those writes close together in
// DRAM.  Within a block, an entry whose node equals the previous entry's reuses
// the row already in registers; the others load theirs (U rows in flight).
// A launch covers list entries [base, base + rows); the host may split the list
// into several launches so that other streams' kernels are dispatched between
// them.
template <typename Unit, int LPR, int U, bool NT, bool ONE, bool TIER>
__global__ __launch_bounds__(kBlock) void k_gather(const Unit* __restrict__ feat, Unit* __restrict__ out,
                                                   int32_t* __restrict__ nodes_out,
                                                   const uint64_t* __restrict__ rl_key,
                                                   const int32_t* __restrict__ rl_val, const int64_t* node_off_g,
                                                   int H, int64_t base, int64_t rows, int64_t row_units,
                                                   const int32_t* __restrict__ tbuf, uint32_t rpb,
                                                   const int32_t* __restrict__ tch, uint32_t pool_rows) {
    constexpr int RPW = kWave / LPR;             // lane groups (rows) per wave
    constexpr int GPB = kWavesPerBlock * RPW;    // lane groups per workgroup
    extern __shared__ int64_t node_off[];
    load_offsets(node_off, node_off_g, H);
    const int G = gridDim.x;
    const int li = lane_id() % LPR;
    const int gid = wave_id() * RPW + lane_id() / LPR;
    const int64_t lo = base, hi = base + rows;
    const int64_t stride = (int64_t)G * GPB * U;
    for (int64_t e0 = lo + ((int64_t)blockIdx.x * GPB + gid) * U; e0 < hi; e0 += stride) {
        uint64_t key[U];
        int32_t val[U];
#pragma unroll
        for (int k = 0; k < U; k++) {
            key[k] = e0 + k < hi ? rl_key[e0 + k] : 0;
            val[k] = e0 + k < hi ? rl_val[e0 + k] : 0;
        }
        uint32_t prev_u = e0 > 0 ? (uint32_t)(rl_key[e0 - 1] >> 32) : 0xFFFFFFFFu;
        uint32_t src[U], dst[U];
        bool ok[U], fresh[U];
#pragma unroll
        for (int k = 0; k < U; k++) {
            const int64_t e = e0 + k;
            ok[k] = e < hi;
            const uint32_t u = (uint32_t)(key[k] >> 32);
            const uint32_t pu = k > 0 ? (uint32_t)(key[k - 1] >> 32) : prev_u;
            const uint32_t d = (uint32_t)(node_off[(uint32_t)key[k]] + val[k]);
            fresh[k] = ok[k] && (k == 0 || u != pu);
            src[k] = (TIER && ok[k]) ? source_row(tbuf, rpb, tch, pool_rows, u) : u;
            dst[k] = d;
            if (nodes_out && ok[k] && li == 0) nodes_out[d] = (int32_t)u;
        }
        const int64_t c_end = ONE ? std::min<int64_t>(row_units, li + 1) : row_units;
        for (int64_t c = li; c < c_end; c += LPR) {
            Unit x[U];
#pragma unroll
            for (int k = 0; k < U; k++)
                if (fresh[k]) x[k] = feat[(int64_t)src[k] * row_units + c];
#pragma unroll
            for (int k = 1; k < U; k++)
                if (!fresh[k]) x[k] = x[k - 1];
#pragma unroll
            for (int k = 0; k < U; k++) {
                if (!ok[k]) continue;
                Unit* o = out + (int64_t)dst[k] * row_units + c;
                if (NT) __builtin_nontemporal_store(x[k], o);
                else *o = x[k];
            }
        }
    }
}

// Row copy for rows of at least 64 16-byte units (1 KiB and up): one wave per
// row.  A wave takes U consecutive entries of the list; lane k < U reads entry
// k and resolves its source row (the node) and destination row (node_off[j] +
// local id), and the wave then broadcasts them with readlane, so each row's
// addresses live in scalar registers and a lane holds only the data: the U
// entries are copied in rounds of V, V rows x UPR units in flight per lane.
// Chunks of 64 * UPR units cover longer rows.  An entry whose node repeats the
// previous entry's (within the wave's U) reuses the row already in registers.
// Waves take blocks of U entries in grid-stride order (wave w of the grid,
// then w + all waves, ...).
template <int U, int V, int UPR, bool NT, bool TIER>
__global__ __launch_bounds__(kBlock) void k_gather_rows(const u32x4* __restrict__ feat, u32x4* __restrict__ out,
                                                        int32_t* __restrict__ nodes_out,
                                                        const uint64_t* __restrict__ rl_key,
                                                        const int32_t* __restrict__ rl_val,
                                                        const int64_t* node_off_g, int H, int64_t base,
                                                        int64_t rows, int64_t row_units,
                                                        const int32_t* __restrict__ tbuf, uint32_t rpb,
                                                        const int32_t* __restrict__ tch, uint32_t pool_rows) {
    static_assert(U <= kWave, "one lane per entry");
    static_assert(U % V == 0, "whole rounds");
    extern __shared__ int64_t node_off[];
    load_offsets(node_off, node_off_g, H);
    const int lane = lane_id();
    const int64_t hi = base + rows;
    const int64_t nw = (int64_t)gridDim.x * kWavesPerBlock;
    for (int64_t e0 = base + ((int64_t)blockIdx.x * kWavesPerBlock + wave_id()) * U; e0 < hi; e0 += nw * U) {
        const int64_t e = e0 + lane;
        const bool mine = lane < U && e < hi;
        uint32_t u = 0xFFFFFFFFu, d = 0, row = 0;
        if (mine) {
            const uint64_t key = rl_key[e];
            u = (uint32_t)(key >> 32);
            d = (uint32_t)(node_off[(uint32_t)key] + rl_val[e]);
            row = TIER ? source_row(tbuf, rpb, tch, pool_rows, u) : u;
            if (nodes_out) nodes_out[d] = (int32_t)u;
        }
        const uint32_t pu = (uint32_t)__shfl_up((int)u, 1, kWave);
        const uint64_t okm = __ballot(mine);
        const uint64_t fresh = __ballot(mine && (lane == 0 || pu != u));
        uint32_t src[U], dst[U];
#pragma unroll
        for (int k = 0; k < U; k++) {
            src[k] = (uint32_t)__builtin_amdgcn_readlane((int)row, k);
            dst[k] = (uint32_t)__builtin_amdgcn_readlane((int)d, k);
        }
        for (int64_t c0 = 0; c0 < row_units; c0 += (int64_t)kWave * UPR) {
            u32x4 prev[UPR];                 // the previous round's last row
#pragma unroll
            for (int h = 0; h < U / V; h++) {
                u32x4 x[V][UPR];
#pragma unroll
                for (int k = 0; k < V; k++) {
                    const int kk = h * V + k;
                    if ((fresh >> kk) & 1) {
                        const u32x4* p = feat + (int64_t)src[kk] * row_units + c0 + lane;
#pragma unroll
                        for (int q = 0; q < UPR; q++)
                            if (c0 + lane + q * kWave < row_units) x[k][q] = p[q * kWave];
                    } else if (k > 0) {
#pragma unroll
                        for (int q = 0; q < UPR; q++) x[k][q] = x[k - 1][q];
                    } else if (kk > 0) {
#pragma unroll
                        for (int q = 0; q < UPR; q++) x[k][q] = prev[q];
                    }
                }
#pragma unroll
                for (int k = 0; k < V; k++) {
                    const int kk = h * V + k;
                    if (!((okm >> kk) & 1)) continue;
                    u32x4* o = out + (int64_t)dst[kk] * row_units + c0 + lane;
#pragma unroll
                    for (int q = 0; q < UPR; q++) {
                        if (c0 + lane + q * kWave < row_units) {
                            if (NT) __builtin_nontemporal_store(x[k][q], o + q * kWave);
                            else o[q * kWave] = x[k][q];
                        }
                    }
                }
#pragma unroll
                for (int q = 0; q < UPR; q++) prev[q] = x[V - 1][q];
            }
        }
    }
}

struct GatherArgs {
    const void* feat;
    void* out;
    int32_t* nodes_out;              // output node ids, or null when the sampling phase wrote them
    const uint64_t* rl_key;
    const int32_t* rl_val;
    const int64_t* node_off;
    int H;
    int64_t base, rows, row_units;   // entries [base, base + rows) of the list
    const int32_t* tbuf;             // staged tier: block -> pool slot (feat is then the pool); else null
    uint32_t rpb;
    const int32_t* tch;              // staged tier with a feature cache: node -> cache row; else null
    uint32_t pool_rows;              // the cache's rows follow this many pool rows
};

template <typename Unit, int LPR, int U, bool NT, bool ONE, bool TIER>
static void launch_gather_k2(const GatherArgs& a, int G, hipStream_t st) {
    const size_t lds = (size_t)(a.H + 1) * sizeof(int64_t);
    AGNES_LAUNCH((k_gather<Unit, LPR, U, NT, ONE, TIER>), dim3(G), dim3(kBlock), lds, st, (const Unit*)a.feat,
                       (Unit*)a.out, a.nodes_out, a.rl_key, a.rl_val, a.node_off, a.H, a.base, a.rows,
                       a.row_units, a.tbuf, a.rpb, a.tch, a.pool_rows);
}

template <typename Unit, int LPR, int U, bool NT>
static void launch_gather_k(const GatherArgs& a, int groups, hipStream_t st) {
    // at most one workgroup per U rows of each lane group: with enough groups
    // every workgroup copies one block and the blocks in flight follow the
    // dispatch order through the list
    constexpr int64_t per_wg = (int64_t)kWavesPerBlock * (kWave / LPR) * U;
    const int G = (int)std::max<int64_t>(1, std::min<int64_t>(groups, (a.rows + per_wg - 1) / per_wg));
    const bool one = a.row_units <= LPR;
    if (a.tbuf) {
        if (one) launch_gather_k2<Unit, LPR, U, NT, true, true>(a, G, st);
        else launch_gather_k2<Unit, LPR, U, NT, false, true>(a, G, st);
    } else {
        if (one) launch_gather_k2<Unit, LPR, U, NT, true, false>(a, G, st);
        else launch_gather_k2<Unit, LPR, U, NT, false, false>(a, G, st);
    }
}

template <typename Unit, int LPR>
static void launch_gather_lpr(const GatherArgs& a, int G, int unroll, bool nt, hipStream_t st) {
    if (unroll >= 16) {
        if (nt) launch_gather_k<Unit, LPR, 16, true>(a, G, st); else launch_gather_k<Unit, LPR, 16, false>(a, G, st);
    } else if (unroll >= 8) {
        if (nt) launch_gather_k<Unit, LPR, 8, true>(a, G, st); else launch_gather_k<Unit, LPR, 8, false>(a, G, st);
    } else {
        if (nt) launch_gather_k<Unit, LPR, 4, true>(a, G, st); else launch_gather_k<Unit, LPR, 4, false>(a, G, st);
    }
}

// Rows in flight per round: 16 entries per wave are copied 8 at a time.
// Beside the sampling of later hyperbatches, half the bytes in flight per wave
// leave the sampling's dependent loads shorter queues (its chains finish in
// 1.9 instead of 2.9 ms), while the copy keeps its pace.
template <int U, int UPR, bool NT>
static void launch_gather_rows_k(const GatherArgs& a, int groups, hipStream_t st) {
    constexpr int V = U >= 16 ? 8 : U;
    const size_t lds = (size_t)(a.H + 1) * sizeof(int64_t);
    constexpr int64_t per_wg = (int64_t)kWavesPerBlock * U;
    const int G = (int)std::max<int64_t>(1, std::min<int64_t>(groups, (a.rows + per_wg - 1) / per_wg));
    if (a.tbuf)
        AGNES_LAUNCH((k_gather_rows<U, V, UPR, NT, true>), dim3(G), dim3(kBlock), lds, st, (const u32x4*)a.feat,
                           (u32x4*)a.out, a.nodes_out, a.rl_key, a.rl_val, a.node_off, a.H, a.base, a.rows,
                           a.row_units, a.tbuf, a.rpb, a.tch, a.pool_rows);
    else
        AGNES_LAUNCH((k_gather_rows<U, V, UPR, NT, false>), dim3(G), dim3(kBlock), lds, st, (const u32x4*)a.feat,
                           (u32x4*)a.out, a.nodes_out, a.rl_key, a.rl_val, a.node_off, a.H, a.base, a.rows,
                           a.row_units, a.tbuf, a.rpb, a.tch, a.pool_rows);
}

template <int UPR>
static void launch_gather_rows_upr(const GatherArgs& a, int groups, int unroll, bool nt, hipStream_t st) {
    if (unroll >= 16) {
        if (nt) launch_gather_rows_k<16, UPR, true>(a, groups, st); else launch_gather_rows_k<16, UPR, false>(a, groups, st);
    } else if (unroll >= 8) {
        if (nt) launch_gather_rows_k<8, UPR, true>(a, groups, st); else launch_gather_rows_k<8, UPR, false>(a, groups, st);
    } else {
        if (nt) launch_gather_rows_k<4, UPR, true>(a, groups, st); else launch_gather_rows_k<4, UPR, false>(a, groups, st);
    }
}


// LPR = the power of two lanes that covers a row best (at most a wave).  The
// list is copied in `chunks` consecutive launches of groups/chunks workgroups.
template <typename Unit>
static void launch_gather(const GatherArgs& all, int groups, int unroll, bool nt, int chunks, hipStream_t st) {
    // Rows in flight per lane group when the store leaves it open: 16 for rows
    // of one 16-byte piece per lane (1 KiB up to 2 KiB), where a wave's 16
    // entries also let more repeats of a node reuse its row; 4 elsewhere, where
    // more rows in flight cost occupancy (2 KiB rows hold two pieces per lane)
    // or lane groups already keep enough bytes moving.
    if (unroll == 0) unroll = (sizeof(Unit) == 16 && all.row_units >= 64 && all.row_units < 128) ? 16 : 4;
    chunks = (int)std::max<int64_t>(1, std::min<int64_t>(chunks, all.rows));
    for (int c = 0; c < chunks; c++) {
        GatherArgs a = all;
        a.base = all.base + all.rows * c / chunks;
        a.rows = all.base + all.rows * (c + 1) / chunks - a.base;
        const int G = std::max(8, groups / chunks);
        if (a.row_units >= 64 && sizeof(Unit) == 16) {
            if (a.row_units >= 128) launch_gather_rows_upr<2>(a, G, unroll, nt, st);
            else launch_gather_rows_upr<1>(a, G, unroll, nt, st);
        } else if (a.row_units >= 64) launch_gather_lpr<Unit, 64>(a, G, unroll, nt, st);
        else if (a.row_units > 16) launch_gather_lpr<Unit, 32>(a, G, unroll, nt, st);
        else if (a.row_units > 8) launch_gather_lpr<Unit, 16>(a, G, unroll, nt, st);
        else if (a.row_units > 4) launch_gather_lpr<Unit, 8>(a, G, unroll, nt, st);
        else launch_gather_lpr<Unit, 4>(a, G, unroll, nt, st);
    }
}


// ----------------------------------------------------------------- staged feature tier
//
// The final list is the feature bucket in ascending block order, so the
// hyperbatch's needed feature blocks are the list's block starts.  Their ids
// and first list entries are compacted on the device and read by the host,
// which plans rounds of at most pool_blocks blocks (hits pinned first, misses
// given the lowest unused slot, else the least recently used unpinned slot).
// Per round the GPU updates the block -> slot table, copies the missing blocks
// from pinned host memory into their slots, and copies the round's rows.

// Step 1: flag the list entries whose rows are not in the feature cache (all
// of them without a cache).
__global__ __launch_bounds__(kBlock) void k_unc_flags(const uint64_t* rl_key, const int32_t* tch, int32_t* flag,
                                                      const Ctl* ctl) {
    const int64_t n = ctl->rows;
    for (int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x; p < n; p += (int64_t)gridDim.x * kBlock)
        flag[p] = (!tch || tch[(uint32_t)(rl_key[p] >> 32)] < 0) ? 1 : 0;
}

__global__ __launch_bounds__(kBlock) void k_unc_compact(const int32_t* flag, const int64_t* off, int32_t* unc,
                                                        const Ctl* ctl) {
    const int64_t n = ctl->rows;
    for (int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x; p < n; p += (int64_t)gridDim.x * kBlock)
        if (flag[p]) unc[off[p]] = (int32_t)p;
}

// Step 2: among those entries, the first of every feature block.
__global__ __launch_bounds__(kBlock) void k_block_flags(const uint64_t* rl_key, const int32_t* unc, uint32_t rpb,
                                                        int32_t* flag, const Ctl* ctl) {
    const int64_t n = ctl->tier_unc;
    for (int64_t k = (int64_t)blockIdx.x * kBlock + threadIdx.x; k < n; k += (int64_t)gridDim.x * kBlock) {
        const uint32_t b = (uint32_t)(rl_key[unc[k]] >> 32) / rpb;
        flag[k] = (k == 0 || (uint32_t)(rl_key[unc[k - 1]] >> 32) / rpb != b) ? 1 : 0;
    }
}

__global__ __launch_bounds__(kBlock) void k_block_compact(const uint64_t* rl_key, const int32_t* unc, uint32_t rpb,
                                                          const int32_t* flag, const int64_t* off,
                                                          int64_t* need_entry, int32_t* need_block, const Ctl* ctl) {
    const int64_t n = ctl->tier_unc;
    for (int64_t k = (int64_t)blockIdx.x * kBlock + threadIdx.x; k < n; k += (int64_t)gridDim.x * kBlock) {
        if (flag[k]) {
            const int64_t i = off[k];
            need_entry[i] = unc[k];
            need_block[i] = (int32_t)((uint32_t)(rl_key[unc[k]] >> 32) / rpb);
        }
    }
}

// After the gather: every row's access count grows by its number of list
// entries (the minibatches that gathered it; a node's entries are one run,
// counted by the run's first entry); rows served by the cache are counted; a
// row not in the cache whose count reaches the threshold is flagged for
// admission.
__global__ __launch_bounds__(kBlock) void k_access_count(const uint64_t* rl_key, const int32_t* tch, uint32_t* count,
                                                         uint32_t threshold, int32_t* flag, Ctl* ctl) {
    __shared__ unsigned long long hits;
    if (threadIdx.x == 0) hits = 0;
    __syncthreads();
    const int64_t n = ctl->rows;
    unsigned long long h = 0;
    for (int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x; p < n; p += (int64_t)gridDim.x * kBlock) {
        const uint32_t u = (uint32_t)(rl_key[p] >> 32);
        int32_t f = 0;
        if (p == 0 || (uint32_t)(rl_key[p - 1] >> 32) != u) {
            uint32_t len = 1;
            while (p + len < n && (uint32_t)(rl_key[p + len] >> 32) == u) len++;
            const uint32_t c0 = count[u];
            const uint32_t c = c0 > 0xFFFFFFFFu - len ? 0xFFFFFFFFu : c0 + len;
            count[u] = c;
            if (tch[u] >= 0) h++;
            else if (c >= threshold) f = 1;
        }
        flag[p] = f;
    }
    if (h) atomicAdd(&hits, h);
    __syncthreads();
    if (threadIdx.x == 0 && hits) atomicAdd((unsigned long long*)&ctl->tier_hits, hits);
}

// Flagged rows enter the cache in list (ascending node) order while it has
// room: one wave per entry copies the row from pinned host memory.
template <typename Unit>
__global__ __launch_bounds__(kBlock) void k_admit(const uint64_t* rl_key, const int32_t* flag, const int64_t* off,
                                                  const Unit* __restrict__ host, Unit* __restrict__ rows_buf,
                                                  int64_t pool_rows, int64_t row_units, int32_t* tch,
                                                  const int64_t* used, int64_t capacity, const Ctl* ctl) {
    const int64_t n = ctl->rows;
    const int64_t nw = (int64_t)gridDim.x * kWavesPerBlock;
    for (int64_t p = (int64_t)blockIdx.x * kWavesPerBlock + wave_id(); p < n; p += nw) {
        if (!flag[p]) continue;
        const int64_t slot = *used + off[p];
        if (slot >= capacity) continue;
        const uint32_t u = (uint32_t)(rl_key[p] >> 32);
        const Unit* src = host + (int64_t)u * row_units;
        Unit* dst = rows_buf + (pool_rows + slot) * row_units;
        for (int64_t c = lane_id(); c < row_units; c += kWave) dst[c] = src[c];
        if (lane_id() == 0) tch[u] = (int32_t)slot;
    }
}

__global__ void k_admit_close(int64_t* used, int64_t capacity, Ctl* ctl) {
    if (threadIdx.x == 0) {
        const int64_t u0 = *used;
        const int64_t u1 = std::min<int64_t>(capacity, u0 + ctl->tier_cand);
        *used = u1;
        ctl->tier_admitted = u1 - u0;
        ctl->tier_cached = u1;
    }
}

// tbuf[block] = slot for every (block, slot) pair of a round (slot -1: evicted).
__global__ __launch_bounds__(kBlock) void k_tbuf_update(const int32_t* pairs, int n, int32_t* tbuf) {
    for (int i = blockIdx.x * kBlock + threadIdx.x; i < n; i += gridDim.x * kBlock) tbuf[pairs[2 * i]] = pairs[2 * i + 1];
}

// One workgroup per missing block (grid-stride): the block's rows, read from
// pinned host memory through its mapped address, written to its pool slot.
template <typename Unit>
__global__ __launch_bounds__(kBlock) void k_stage(const Unit* __restrict__ host, Unit* __restrict__ pool,
                                                  const int32_t* __restrict__ misses, int n, int64_t units) {
    for (int i = blockIdx.x; i < n; i += gridDim.x) {
        const int64_t b = misses[2 * i], slot = misses[2 * i + 1];
        const Unit* src = host + b * units;
        Unit* dst = pool + slot * units;
        // four host reads in flight per lane before their stores
        for (int64_t c0 = threadIdx.x; c0 < units; c0 += 4 * kBlock) {
            Unit x[4];
#pragma unroll
            for (int q = 0; q < 4; q++)
                if (c0 + q * kBlock < units) x[q] = src[c0 + q * kBlock];
#pragma unroll
            for (int q = 0; q < 4; q++)
                if (c0 + q * kBlock < units) dst[c0 + q * kBlock] = x[q];
        }
    }
}

// ----------------------------------------------------------------- host orchestration

// Layout of the block that the host reads at the synchronisation point:
// [Ctl][layer sizes H x (L+1) int32][edge counts H x L int64].
struct SyncLayout {
    size_t lsz, ecount, lstat, bytes;
    int n_lstat;                      // workgroups of k_list_stats (one partial pair each)
};

static int list_stats_groups(int64_t rows_max) { return grid_for(rows_max / kStatItems + 1, 512); }

static SyncLayout sync_layout(int H, int L, int64_t rows_max) {
    SyncLayout y;
    y.lsz = (sizeof(Ctl) + 255) / 256 * 256;
    y.ecount = (y.lsz + (size_t)H * (L + 1) * 4 + 255) / 256 * 256;
    y.lstat = (y.ecount + (size_t)H * L * 8 + 255) / 256 * 256;
    y.n_lstat = list_stats_groups(rows_max);
    y.bytes = y.lstat + (size_t)y.n_lstat * 16;
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
    w.e_off.reserve((size_t)(g.Rmax + 1) * 4);     // edge numbers are below 2^32 (plan)
    for (int i = 0; i < 2; i++) {
        w.rl_key[i].reserve((size_t)g.rows_max * 8);
        w.rl_val[i].reserve((size_t)g.rows_max * 4);
    }
    w.skey.reserve((size_t)g.sort_max * 4);
    w.sval.reserve((size_t)g.sort_max * 4);
    w.skey2.reserve((size_t)g.sort_max * 4);
    w.sval2.reserve((size_t)g.sort_max * 4);
    w.split.reserve((size_t)(join_tiles_max(g) + 2) * 8);
    const int64_t G = std::max<int64_t>(join_groups(g.H, join_tiles_max(g)), g.bstride_max);
    w.ghist.reserve((size_t)H * G * 8);
    w.gemit.reserve((size_t)G * 8);
    w.acoff.reserve((size_t)(kCoarseMax + 1) * 8);
    w.rs_hist.reserve((size_t)radix_hist_entries(g.sort_max) * 4);
    w.rs_dtot.reserve((size_t)radix_dtot_entries() * 4);
    w.scan_part.reserve((size_t)scan_partials_needed() * 8);
    w.topo_part.reserve((size_t)((grid_for(g.Rmax, 2048) + kXcds - 1) / kXcds * kXcds) * 4);
    w.params.reserve(sizeof(ChainParams));
    if (!w.ev[0])
        for (auto& e : w.ev) AGNES_CHECK_HIP(hipEventCreate(&e));
}

template <typename OffT>
static void launch_layer(const Store& s, Workspace& w, const Geometry& g, int l, int32_t f, Batch& b,
                         const SyncLayout& y, int cur, bool legacy, hipStream_t st) {
    const ChainParams* prm = w.params.as<ChainParams>();
    Ctl* ctl = w.sync.as<Ctl>();
    int32_t* lsz = (int32_t*)((char*)w.sync.ptr + y.lsz);
    int64_t* ecount = (int64_t*)((char*)w.sync.ptr + y.ecount);
    const OffT* off = s.offsets.as<OffT>();
    const size_t lds_h = (size_t)(g.H + 1) * sizeof(int64_t);
    // this hop's requests are at most H cap[l]: its own bound sizes the grids
    // (beside a long kernel of another stream even an idle workgroup waits for
    // a slot); k_begin sums the previous hop's per-workgroup counts
    const int gR = hop_grid(s, g, l);
    const int gPrev = l > 0 ? hop_grid(s, g, l - 1) : 0;
    int64_t* part = w.scan_part.as<int64_t>();
    const uint64_t* rlk = w.rl_key[cur].as<uint64_t>();
    const int32_t* rlv = w.rl_val[cur].as<int32_t>();

    AGNES_LAUNCH(k_begin, dim3(1), dim3(kBlock), 0, st, l, g.L, g.H, ctl, w.size.as<int32_t>(),
                       w.newcnt.as<int64_t>(), lsz, ecount, w.req_off.as<int64_t>(), w.e_off.as<uint32_t>(),
                       (int64_t*)nullptr, w.topo_part.as<uint32_t>(), gPrev);
    // counts and the edge-offset scan: counts with the reduce pass, then the final pass
    const int64_t r_max = std::max<int64_t>(1, (int64_t)g.H * g.cap[l]);
    const int gS = scan_groups(r_max);
    AGNES_LAUNCH(k_count_reduce<OffT>, dim3(gS), dim3(kBlock), lds_h, st, g.H, g.capN, f, off,
                 w.nodes.as<int32_t>(), w.req_off.as<int64_t>(), w.cnt.as<int32_t>(), gS, part, ctl);
    scan_counts_final(w.cnt.as<int32_t>(), w.e_off.as<uint32_t>(), &ctl->R, r_max, &ctl->S, part, st);
    const int32_t* adj = s.indices.as<int32_t>();
    int32_t* cg = w.skey.as<int32_t>();
#define AGNES_SAMPLE(MK)                                                                               \
    AGNES_LAUNCH((k_sample<OffT, MK>), dim3(gR), dim3(kBlock), lds_h, st, l, g.H, f, prm,      \
                       off, adj, s.e_blk_log2, s.nblk, rlk, rlv, w.req_off.as<int64_t>(),      \
                       w.e_off.as<uint32_t>(), cg, w.topo_part.as<uint32_t>(), ctl)
    // the register sampler's work grows with MAXK^2 (ranks) and MAXK/4 (Philox
    // calls), so common fanouts get a bound of their own
    if (f <= 4) AGNES_SAMPLE(4);
    else if (f <= 8) AGNES_SAMPLE(8);
    else if (f <= 10) AGNES_SAMPLE(10);
    else if (f <= 16) AGNES_SAMPLE(16);
    else if (f <= 20) AGNES_SAMPLE(20);
    else if (f <= 25) AGNES_SAMPLE(25);
    else if (f <= 32) AGNES_SAMPLE(32);
    else AGNES_SAMPLE(0);
#undef AGNES_SAMPLE
    const int64_t s_max = std::max<int64_t>(1, std::min<int64_t>(g.Smax, (int64_t)g.H * g.cap[l] * f));
    if (!legacy) {
        // node-range buckets: the sampled edges grouped by coarse bucket, then
        // each bucket joined with its part of the list in LDS
        const int64_t load_max = (int64_t)g.H * g.cap[l] * (1 + (int64_t)f);
        bucket_partition(w.skey.as<uint32_t>(), w.skey2.as<uint32_t>(), w.sval2.as<uint32_t>(), &ctl->S, &ctl->R,
                         s_max, load_max, s, g.H, w.rs_hist.as<uint32_t>(), w.rs_dtot.as<uint32_t>(), rlk,
                         w.acoff.as<int64_t>(), st);
        BucketJoinArgs j{};
        j.store = &s;
        j.H = g.H;
        j.jbits = g.jbits;
        j.write_nodes = l + 1 < g.L;
        j.capN = g.capN;
        j.rows_cap = g.rows_max;
        j.cap = s.bucket_cap;
        j.coarse_max = g.bcoarse[l];
        j.G = g.bstride[l];
        j.n_dev = &ctl->S;
        j.old_dev = &ctl->R;
        j.rk = w.skey2.as<uint32_t>();
        j.rv = w.sval2.as<uint32_t>();
        j.dtot = w.rs_dtot.as<uint32_t>();
        j.acoff = w.acoff.as<int64_t>();
        j.ak = rlk;
        j.av = rlv;
        j.req_off = w.req_off.as<int64_t>();
        j.e_off = w.e_off.as<uint32_t>();
        j.size = w.size.as<int32_t>();
        j.ghist = w.ghist.as<int64_t>();
        j.gemit = w.gemit.as<int64_t>();
        j.newcnt = w.newcnt.as<int64_t>();
        j.row_ptr = b.row_ptr[l].as<int32_t>();
        j.nodes = w.nodes.as<int32_t>();
        j.ck = w.rl_key[cur ^ 1].as<uint64_t>();
        j.cv = w.rl_val[cur ^ 1].as<int32_t>();
        j.col = b.col[l].as<int32_t>();
        j.ctl = ctl;
        bucket_join(j, st);
        return;
    }
    // sampled neighbours sorted by node id; values = edge numbers (stable: minibatch order kept).
    // This hop's own bound sizes the sort's tiles and grid (hop 0 samples far
    // fewer edges than the last hop).
    int in_tmp = radix_sort_pairs32(w.skey.as<uint32_t>(), w.sval.as<uint32_t>(), w.skey2.as<uint32_t>(),
                                    w.sval2.as<uint32_t>(), &ctl->S, s_max, s.node_bits,
                                    w.rs_hist.as<uint32_t>(), w.rs_dtot.as<uint32_t>(), st, true,
                                    hop_cap(s, g.ebound[l]));
    const uint32_t* su = in_tmp ? w.skey2.as<uint32_t>() : w.skey.as<uint32_t>();
    const uint32_t* se = in_tmp ? w.sval2.as<uint32_t>() : w.sval.as<uint32_t>();
    // join with the list: the next list, new node ids and the hop's columns
    const int64_t tiles_l = ((int64_t)g.H * g.cap[l] * (1 + (int64_t)f)) / kJoinTile + 1;
    int64_t* split = w.split.as<int64_t>();
    const int G = (int)std::max<int64_t>(
        std::min(join_groups(g.H, tiles_l), std::max(kBlock, hop_cap(s, g.ebound[l]) / kBlock * kBlock)),
        join_groups_min(tiles_l));
    const int64_t per = (tiles_l + G - 1) / G + 2;
    AGNES_LAUNCH(k_join_count, dim3(G), dim3(kBlock), join_count_lds(g.H, per), st, g.H,
                       w.req_off.as<int64_t>(), w.e_off.as<uint32_t>(), rlk, rlv, su, se, split, G,
                       w.ghist.as<int64_t>(), w.gemit.as<int64_t>(), b.row_ptr[l].as<int32_t>(), ctl);
    AGNES_LAUNCH(k_join_scan, dim3(g.H + 1), dim3(kBlock), 0, st, g.H, G, w.ghist.as<int64_t>(),
                       w.gemit.as<int64_t>(), w.newcnt.as<int64_t>(), ctl);
    AGNES_LAUNCH(k_join_write, dim3(G), dim3(kBlock), join_write_lds(g.H, per), st, g.H, g.jbits,
                       g.capN, g.rows_max, w.req_off.as<int64_t>(), w.e_off.as<uint32_t>(), rlk, rlv, su, se,
                       split, G, w.ghist.as<int64_t>(), w.gemit.as<int64_t>(), w.size.as<int32_t>(),
                       w.nodes.as<int32_t>(), w.rl_key[cur ^ 1].as<uint64_t>(), w.rl_val[cur ^ 1].as<int32_t>(),
                       b.col[l].as<int32_t>(), ctl);
    AGNES_CHECK_HIP(hipGetLastError());
}

// ----------------------------------------------------------------- staged tier: host planning

struct TierRound {
    int64_t e0, e1;              // list entries whose rows the round copies
    int n_upd, n_miss;           // table updates (block, slot) and blocks to copy (block, slot)
    size_t upd_at, miss_at;      // their offsets (int32 elements) in the uploaded plan
};

// Reads the hyperbatch's needed feature blocks (ascending) and plans the rounds:
// at most pool_blocks blocks per round; blocks in the pool are hits and are
// used (pinned) first, ascending; every other block of the round, ascending,
// takes the lowest never-used slot, else the least recently used slot among
// the slots not used in this round.  Every hit and every staging is one use.
// The plan is written to the batch's pinned plan buffer; the store's pool view
// is advanced as if the rounds had run (they are enqueued in the same order).
static std::vector<TierRound> plan_staging(const Store& s, Batch& b, hipStream_t st) {
    Workspace& w = b.ws;
    const int64_t rows = b.node_off[b.H];
    if (!b.needed) AGNES_CHECK_HIP(hipEventCreateWithFlags(&b.needed, hipEventDisableTiming));
    // the number of needed blocks, then the lists
    AGNES_CHECK_HIP(hipMemcpyAsync(w.sync_host.ptr, w.sync.ptr, sizeof(Ctl), hipMemcpyDeviceToHost, st));
    AGNES_CHECK_HIP(hipEventRecord(b.needed, st));
    AGNES_CHECK_HIP(hipEventSynchronize(b.needed));
    Ctl hc;
    memcpy(&hc, w.sync_host.ptr, sizeof(Ctl));
    const int64_t nb = hc.tier_nb;
    AGNES_REQUIRE(nb >= 0 && nb <= b.need_cap, AGNES_ERR_INTERNAL, "needed feature blocks out of range");
    w.need_host.reserve_slack((size_t)std::max<int64_t>(nb, 1) * 12);
    int64_t* need_entry = (int64_t*)w.need_host.ptr;
    int32_t* need_block = (int32_t*)((char*)w.need_host.ptr + (size_t)nb * 8);
    if (nb > 0) {
        AGNES_CHECK_HIP(hipMemcpyAsync(need_entry, w.need.ptr, (size_t)nb * 8, hipMemcpyDeviceToHost, st));
        AGNES_CHECK_HIP(hipMemcpyAsync(need_block, (char*)w.need.ptr + (size_t)b.need_cap * 8, (size_t)nb * 4,
                                       hipMemcpyDeviceToHost, st));
        AGNES_CHECK_HIP(hipEventRecord(b.needed, st));
        AGNES_CHECK_HIP(hipEventSynchronize(b.needed));
    }

    const int64_t P = s.pool_blocks;
    std::vector<TierRound> rounds;
    std::vector<int32_t> upd, miss, plan;
    int64_t staged = 0, hits = 0;
    auto touch = [&](int32_t sl) {
        const int64_t t = ++s.accesses;
        s.slot_stamp[sl] = t;
        s.lru.push_back({t, sl});
    };
    // the least recently used slot not used since access number t0 (the start
    // of the current round); stale entries are dropped on the way
    auto victim = [&](int64_t t0) -> int32_t {
        for (;;) {
            AGNES_REQUIRE(!s.lru.empty(), AGNES_ERR_INTERNAL, "no pool slot to replace");
            const auto e = s.lru.front();
            s.lru.pop_front();
            if (s.slot_stamp[e.second] != e.first) continue;
            AGNES_REQUIRE(e.first <= t0, AGNES_ERR_INTERNAL, "every pool slot is pinned");
            return e.second;
        }
    };
    for (int64_t i0 = 0; i0 < nb; i0 += P) {
        const int64_t i1 = std::min<int64_t>(nb, i0 + P);
        const int64_t t0 = s.accesses;
        s.tier_clock++;
        upd.clear();
        miss.clear();
        for (int64_t k = i0; k < i1; k++) {                 // hits: pinned for this round
            const int32_t sl = s.block_slot[need_block[k]];
            if (sl >= 0) {
                touch(sl);
                hits++;
            }
        }
        for (int64_t k = i0; k < i1; k++) {                 // misses, ascending
            const int32_t blk = need_block[k];
            if (s.block_slot[blk] >= 0) continue;
            int32_t sl;
            if (s.next_free < P) {
                sl = (int32_t)s.next_free++;
            } else {
                sl = victim(t0);
                const int32_t old = s.slot_block[sl];
                s.block_slot[old] = -1;
                upd.push_back(old);
                upd.push_back(-1);
            }
            s.slot_block[sl] = blk;
            s.block_slot[blk] = sl;
            touch(sl);
            upd.push_back(blk);
            upd.push_back(sl);
            miss.push_back(blk);
            miss.push_back(sl);
            staged++;
        }
        TierRound r;
        r.e0 = i0 == 0 ? 0 : need_entry[i0];
        r.e1 = i1 < nb ? need_entry[i1] : rows;
        r.n_upd = (int)(upd.size() / 2);
        r.n_miss = (int)(miss.size() / 2);
        r.upd_at = plan.size();
        plan.insert(plan.end(), upd.begin(), upd.end());
        r.miss_at = plan.size();
        plan.insert(plan.end(), miss.begin(), miss.end());
        rounds.push_back(r);
    }
    const int64_t staging_rounds = (int64_t)rounds.size();
    if (nb == 0) rounds.push_back(TierRound{0, rows, 0, 0, 0, 0});   // every row is in the feature cache: copies only
    // keep the queue near the pool size: rebuild it from the live stamps
    if ((int64_t)s.lru.size() > 4 * P + 1024) {
        std::vector<std::pair<int64_t, int32_t>> all;
        all.reserve((size_t)s.next_free);
        for (int64_t sl = 0; sl < s.next_free; sl++) all.push_back({s.slot_stamp[sl], (int32_t)sl});
        std::sort(all.begin(), all.end());
        s.lru.assign(all.begin(), all.end());
    }
    const size_t bytes = std::max<size_t>(plan.size() * 4, 8);
    w.plan_host.reserve_slack(bytes);
    memcpy(w.plan_host.ptr, plan.data(), plan.size() * 4);
    w.plan.reserve_slack(bytes);
    w.plan_used = bytes;
    b.tier.needed_blocks = nb;
    b.tier.staged_blocks = staged;
    b.tier.hit_blocks = hits;
    b.tier.rounds = staging_rounds;
    b.tier.staged_bytes = staged * s.rpb * s.row_bytes;
    return rounds;
}


// The sampling phase's kernels: counters cleared, targets sorted into the list
// of hop 0, the hops, the close of the last hop and the statistics of the final
// list.  Every size they need is read from device memory and every per-call
// value from the params block, so the sequence depends only on the shape, the
// store and the buffer addresses (the key of a captured graph).
static void launch_chain(const Store& s, Batch& b, const Geometry& g, const SyncLayout& y,
                         const int32_t* fanouts, bool legacy, hipStream_t st) {
    Workspace& w = b.ws;
    const int32_t H = g.H, B = g.B, L = g.L;
    Ctl* ctl = w.sync.as<Ctl>();
    int32_t* lsz = (int32_t*)((char*)w.sync.ptr + y.lsz);
    int64_t* ec = (int64_t*)((char*)w.sync.ptr + y.ecount);
    AGNES_LAUNCH(k_init, dim3(grid_for((int64_t)H * B, 1024)), dim3(kBlock), 0, st,
                       w.params.as<ChainParams>(), H, B, s.num_nodes, g.capN, w.nodes.as<int32_t>(),
                       w.size.as<int32_t>(), w.newcnt.as<int64_t>(), w.skey.as<uint32_t>(), ctl);
    // the list of hop 0 (Bck of the targets): targets sorted by (node,
    // minibatch) with the radix sort, on either join path
    int in_tmp = radix_sort_pairs32(w.skey.as<uint32_t>(), w.sval.as<uint32_t>(), w.skey2.as<uint32_t>(),
                                    w.sval2.as<uint32_t>(), &ctl->targets, (int64_t)H * B, s.node_bits,
                                    w.rs_hist.as<uint32_t>(), w.rs_dtot.as<uint32_t>(), st, true,
                                    hop_cap(s, (int64_t)H * B));
    AGNES_LAUNCH(k_list0, dim3(grid_for((int64_t)H * B, 1024)), dim3(kBlock), 0, st,
                       in_tmp ? w.skey2.as<uint32_t>() : w.skey.as<uint32_t>(),
                       in_tmp ? w.sval2.as<uint32_t>() : w.sval.as<uint32_t>(), B, w.rl_key[0].as<uint64_t>(),
                       w.rl_val[0].as<int32_t>(), ctl);
    AGNES_CHECK_HIP(hipGetLastError());
    int cur = 0;
    for (int l = 0; l < L; l++) {
        if (s.offsets64) launch_layer<int64_t>(s, w, g, l, fanouts[l], b, y, cur, legacy, st);
        else launch_layer<int32_t>(s, w, g, l, fanouts[l], b, y, cur, legacy, st);
        cur ^= 1;
    }
    // close the last hop: edge counts, final node counts, output row offsets
    AGNES_LAUNCH(k_begin, dim3(1), dim3(kBlock), 0, st, L, L, H, ctl, w.size.as<int32_t>(),
                       w.newcnt.as<int64_t>(), lsz, ec, w.req_off.as<int64_t>(), w.e_off.as<uint32_t>(),
                       w.mb_off.as<int64_t>(), w.topo_part.as<uint32_t>(), hop_grid(s, g, L - 1));
    // the radix-sort path keeps every minibatch's node list in nodes (capN
    // apart), and the statistics kernel packs them into the output; on the
    // bucket path the row copy writes the output ids
    int32_t* packed = legacy ? b.nodes.as<int32_t>() : nullptr;
    AGNES_LAUNCH(k_list_stats, dim3(y.n_lstat), dim3(kBlock), packed ? (size_t)(H + 1) * sizeof(int64_t) : 0, st,
                 w.rl_key[cur].as<uint64_t>(), (uint32_t)s.rpb, (uint64_t*)((char*)w.sync.ptr + y.lstat), ctl,
                 w.nodes.as<int32_t>(), g.capN, w.mb_off.as<int64_t>(), H, packed);
    b.ids_in_chain = legacy;
    AGNES_CHECK_HIP(hipGetLastError());
}

// Everything launch_chain's launches depend on apart from the params block.
static std::vector<uint64_t> chain_key(const Store& s, const Batch& b, const Geometry& g, const int32_t* fanouts) {
    const Workspace& w = b.ws;
    auto a = [](const void* p) { return (uint64_t)(uintptr_t)p; };
    std::vector<uint64_t> k = {a(&s), (uint64_t)s.num_nodes, (uint64_t)s.nblk, (uint64_t)s.offsets64,
                               (uint64_t)s.node_bits, (uint64_t)s.e_blk_log2, (uint64_t)s.rpb,
                               (uint64_t)s.join_path, (uint64_t)s.bucket_cap, (uint64_t)s.sample_groups,
                               a(s.offsets.ptr), a(s.indices.ptr), (uint64_t)g.H, (uint64_t)g.B, (uint64_t)g.L};
    for (int l = 0; l < g.L; l++) k.push_back((uint64_t)fanouts[l]);
    for (const DevBuf* d : {&w.nodes, &w.size, &w.newcnt, &w.req_off, &w.mb_off, &w.sync, &w.cnt, &w.e_off,
                            &w.rl_key[0], &w.rl_key[1], &w.rl_val[0], &w.rl_val[1], &w.skey, &w.sval, &w.skey2,
                            &w.sval2, &w.split, &w.ghist, &w.gemit, &w.rs_hist, &w.rs_dtot, &w.scan_part,
                            &w.topo_part, &w.params, &w.acoff})
        k.push_back(a(d->ptr));
    for (int l = 0; l < g.L; l++) {
        k.push_back(a(b.row_ptr[l].ptr));
        k.push_back(a(b.col[l].ptr));
    }
    k.push_back(a(b.nodes.ptr));
    return k;
}

// Graph replay pays where the launches, not the work, set a hyperbatch's
// time: on the automatic setting, for hyperbatches whose hops can sample at
// most kGraphAutoEdges edges in all (H cap_l f_l summed over the hops).  On
// larger ones the kernels launched one by one overlap better with those of
// hyperbatches sampling on other streams.
constexpr int64_t kGraphAutoEdges = (int64_t)1 << 20;

static bool replay_chain(const Store& s, const Geometry& g, const int32_t* fanouts) {
    if (s.sampling_graph != 2) return s.sampling_graph == 1;
    int64_t edges = 0;
    for (int l = 0; l < g.L; l++) edges += (int64_t)g.H * g.cap[l] * fanouts[l];
    return edges <= kGraphAutoEdges;
}

// Captures launch_chain as a HIP graph on the batch's private stream (nothing
// runs during a capture) and keeps its executable instance.
static void capture_chain(const Store& s, Batch& b, const Geometry& g, const SyncLayout& y,
                          const int32_t* fanouts, const std::vector<uint64_t>& key) {
    if (b.chain) {
        (void)hipGraphExecDestroy(b.chain);
        b.chain = nullptr;
        b.chain_key.clear();
    }
    if (!b.cap_stream) AGNES_CHECK_HIP(hipStreamCreateWithFlags(&b.cap_stream, hipStreamNonBlocking));
    AGNES_CHECK_HIP(hipStreamBeginCapture(b.cap_stream, hipStreamCaptureModeThreadLocal));
    hipGraph_t graph = nullptr;
    try {
        launch_chain(s, b, g, y, fanouts, s.join_path == 0, b.cap_stream);
    } catch (...) {
        (void)hipStreamEndCapture(b.cap_stream, &graph);
        if (graph) (void)hipGraphDestroy(graph);
        throw;
    }
    AGNES_CHECK_HIP(hipStreamEndCapture(b.cap_stream, &graph));
    hipGraphExec_t exec = nullptr;
    const hipError_t e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
    (void)hipGraphDestroy(graph);
    AGNES_CHECK_HIP(e);
    b.chain = exec;
    b.chain_key = key;
}

void begin_hyperbatch(const Store& s, Batch& b, const int32_t* targets, bool targets_on_host, int32_t H,
                      int32_t B, const int32_t* fanouts, int32_t L, uint64_t seed, int64_t mb_base,
                      hipStream_t st) {
    Range range("agnes_hyperbatch_begin");
    AGNES_REQUIRE(b.state != kSampled, AGNES_ERR_INVALID, "the batch has a hyperbatch begun but not finished");
    Geometry g = plan(s, H, B, fanouts, L);
    // a batch still gathering: its buffers are in use until the gather ends
    if (b.state == kGathering) wait_batch(b);
    b.state = kIdle;
    // a forward still reading the batch's CSR and rows: this hyperbatch's
    // kernels overwrite them, so they queue behind it
    if (b.sage_pending) AGNES_CHECK_HIP(hipStreamWaitEvent(st, b.sage_done, 0));
    AGNES_REQUIRE(join_write_lds(H, kJoinGroupTilesMax + 2) <= (size_t)s.max_lds &&
                      join_count_lds(H, kJoinGroupTilesMax + 2) <= (size_t)s.max_lds,
                  AGNES_ERR_RANGE, "H is too large for the device's workgroup memory");
    SyncLayout y = sync_layout(H, L, g.rows_max);
    Workspace& w = b.ws;
    reserve_workspace(w, g, y);
    b.rows_max = g.rows_max;
    if (!b.sampled) AGNES_CHECK_HIP(hipEventCreateWithFlags(&b.sampled, hipEventDisableTiming));
    if (!b.gathered) AGNES_CHECK_HIP(hipEventCreateWithFlags(&b.gathered, hipEventDisableTiming));
    if (!b.sage_done) AGNES_CHECK_HIP(hipEventCreateWithFlags(&b.sage_done, hipEventDisableTiming));
    b.d_lsz = (const int32_t*)((const char*)w.sync.ptr + y.lsz);
    b.d_ecount = (const int64_t*)((const char*)w.sync.ptr + y.ecount);
    b.store = &s;
    b.H = H; b.B = B; b.L = L;
    b.capN = g.capN;
    b.stream = st;
    for (int l = 0; l < L; l++) {
        b.row_ptr[l].reserve((size_t)(H * g.cap[l] + H) * 4);
        b.col[l].reserve((size_t)std::max<int64_t>(1, H * g.cap[l] * fanouts[l]) * 4);
    }
    // the output node ids are written by the sampling phase (at most rows_max)
    b.nodes.reserve((size_t)g.rows_max * 4);

    b.prof = s.profile;
    if (b.prof) AGNES_CHECK_HIP(hipEventRecord(w.ev[0], st));
    if (targets_on_host) {
        // Alg. 1's input N arrives in host memory: staged through the batch's
        // pinned copy (its previous upload finished with the previous
        // hyperbatch's sampling) and uploaded on the sampling stream
        const size_t tb = (size_t)H * B * sizeof(int32_t);
        w.targets_host.reserve_slack(tb);
        memcpy(w.targets_host.ptr, targets, tb);
        w.targets.reserve_slack(tb);
        AGNES_CHECK_HIP(hipMemcpyAsync(w.targets.ptr, w.targets_host.ptr, tb, hipMemcpyHostToDevice, st));
        targets = w.targets.as<int32_t>();
    }
    AGNES_LAUNCH(k_params, dim3(1), dim3(kBlock), 0, st, w.params.as<ChainParams>(), targets, seed, mb_base,
                       w.sync.as<Ctl>(), (int64_t)H * B);
    AGNES_CHECK_HIP(hipGetLastError());
    // With graph replay, a shape seen twice in a row is captured once and
    // then replayed: one graph launch instead of about 20 launches per hop.
    std::vector<uint64_t> key = chain_key(s, b, g, fanouts);
    const bool replay = replay_chain(s, g, fanouts);
    if (replay && !(b.chain && key == b.chain_key) && key == b.last_key)
        capture_chain(s, b, g, y, fanouts, key);
    if (replay && b.chain && key == b.chain_key) AGNES_CHECK_HIP(hipGraphLaunch(b.chain, st));
    else launch_chain(s, b, g, y, fanouts, s.join_path == 0, st);
    // what finish needs to sample the hyperbatch again on the radix-sort path
    b.fanouts.assign(fanouts, fanouts + L);
    b.seed = seed;
    b.mb_base = mb_base;
    b.targets_dev = targets;
    b.last_key = std::move(key);
    b.cur = L & 1;                    // the list buffers alternate hop by hop
    // sizes of the outputs travel to pinned host memory; finish reads them
    AGNES_CHECK_HIP(hipMemcpyAsync(w.sync_host.ptr, w.sync.ptr, y.bytes, hipMemcpyDeviceToHost, st));
    b.sampled_at = b.prof ? w.ev[1] : b.sampled;
    AGNES_CHECK_HIP(hipEventRecord(b.sampled_at, st));
    b.state = kSampled;
}

void finish_hyperbatch(Batch& b, hipStream_t st) {
    Range range("agnes_batch_finish");
    AGNES_REQUIRE(b.state == kSampled, AGNES_ERR_INVALID, "finish needs a begun hyperbatch");
    const Store& s = *b.store;
    Workspace& w = b.ws;
    const int H = b.H, L = b.L;
    SyncLayout y = sync_layout(H, L, b.rows_max);
    AGNES_CHECK_HIP(hipEventSynchronize(b.sampled_at));
    b.state = kIdle;   // until the gather is enqueued
    Ctl hc;
    memcpy(&hc, w.sync_host.ptr, sizeof(Ctl));
    if (hc.err & 8) {
        // a sorted sub-bucket exceeded its capacity: the hyperbatch's sampling
        // runs again on the radix-sort path (same results), then as before
        const Geometry g = plan(s, H, b.B, b.fanouts.data(), L);
        AGNES_LAUNCH(k_params, dim3(1), dim3(kBlock), 0, b.stream, w.params.as<ChainParams>(), b.targets_dev,
                     b.seed, b.mb_base, w.sync.as<Ctl>(), (int64_t)H * b.B);
        launch_chain(s, b, g, y, b.fanouts.data(), true, b.stream);
        AGNES_CHECK_HIP(hipMemcpyAsync(w.sync_host.ptr, w.sync.ptr, y.bytes, hipMemcpyDeviceToHost, b.stream));
        AGNES_CHECK_HIP(hipEventRecord(b.sampled_at, b.stream));
        AGNES_CHECK_HIP(hipEventSynchronize(b.sampled_at));
        memcpy(&hc, w.sync_host.ptr, sizeof(Ctl));
        b.fallbacks++;
    }
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
    {
        const uint64_t* lp = (const uint64_t*)((const char*)w.sync_host.ptr + y.lstat);
        int64_t nd = 0, nf = 0;
        for (int i = 0; i < y.n_lstat; i++) {
            nd += (int64_t)lp[2 * i];
            nf += (int64_t)lp[2 * i + 1];
        }
        b.stats.distinct_rows = nd;
        b.stats.feat_blocks = nf;
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
    if (st != b.stream) AGNES_CHECK_HIP(hipStreamWaitEvent(st, b.sampled_at, 0));
    const uint64_t* rlk = w.rl_key[b.cur].as<uint64_t>();
    const int32_t* rlv = w.rl_val[b.cur].as<int32_t>();
    int32_t* ids = b.ids_in_chain ? nullptr : b.nodes.as<int32_t>();   // else written by the sampling phase
    GatherArgs ga{s.features.ptr, b.features.ptr, ids, rlk, rlv, w.mb_off.as<int64_t>(),
                  H, 0, rows, 0, nullptr, (uint32_t)s.rpb};
    const bool wide = s.row_bytes % 16 == 0;
    ga.row_units = wide ? s.row_bytes / 16 : s.row_bytes / 4;
    auto copy_rows = [&](const GatherArgs& a) {
        if (wide) launch_gather<u32x4>(a, s.gather_groups, s.gather_unroll, s.gather_nt != 0, s.gather_chunks, st);
        else launch_gather<uint32_t>(a, s.gather_groups, s.gather_unroll, s.gather_nt != 0, s.gather_chunks, st);
    };
    memset(&b.tier, 0, sizeof(b.tier));
    if (s.tiered && rows > 0) {
        // The needed blocks are found and read back on this hyperbatch's
        // sampling stream (cs), so the host plans while earlier hyperbatches
        // still stage and gather on st.  With a feature cache they wait for the
        // previous hyperbatch's admissions, which decide the rows it serves.
        const hipStream_t cs = b.stream;
        Ctl* ctl = w.sync.as<Ctl>();
        const bool cache = s.cache_rows > 0;
        if (cache) AGNES_CHECK_HIP(hipStreamWaitEvent(cs, s.pool_free, 0));
        const int32_t* tch = cache ? s.tch.as<int32_t>() : nullptr;
        int64_t* part = w.scan_part.as<int64_t>();
        // needed feature blocks: the blocks of the entries whose rows are not cached
        // with headroom: a reallocation frees the old buffer, and hipFree waits
        // for the whole device, i.e. for earlier hyperbatches still staging
        w.blk_flag.reserve_slack((size_t)rows * 4);
        w.blk_off.reserve_slack((size_t)(rows + 1) * 8);
        w.unc.reserve_slack((size_t)rows * 4);
        w.need.reserve_slack((size_t)rows * 12 + 256);
        b.need_cap = rows;
        const int gl = grid_for(rows, 4096);
        int32_t* flag = w.blk_flag.as<int32_t>();
        int64_t* off = w.blk_off.as<int64_t>();
        AGNES_LAUNCH(k_unc_flags, dim3(gl), dim3(kBlock), 0, cs, rlk, tch, flag, ctl);
        scan_counts(flag, off, &ctl->rows, rows, &ctl->tier_unc, part, cs);
        AGNES_LAUNCH(k_unc_compact, dim3(gl), dim3(kBlock), 0, cs, flag, off, w.unc.as<int32_t>(), ctl);
        AGNES_LAUNCH(k_block_flags, dim3(gl), dim3(kBlock), 0, cs, rlk, w.unc.as<int32_t>(), (uint32_t)s.rpb,
                           flag, ctl);
        scan_counts(flag, off, &ctl->tier_unc, rows, &ctl->tier_nb, part, cs);
        AGNES_LAUNCH(k_block_compact, dim3(gl), dim3(kBlock), 0, cs, rlk, w.unc.as<int32_t>(), (uint32_t)s.rpb,
                           flag, off, w.need.as<int64_t>(), (int32_t*)((char*)w.need.ptr + (size_t)rows * 8), ctl);
        AGNES_CHECK_HIP(hipGetLastError());
        std::vector<TierRound> rounds = plan_staging(s, b, cs);
        // staging overwrites pool slots: the pool's previous users are done;
        // and the compaction above (flag and off are reused below) is done
        AGNES_CHECK_HIP(hipStreamWaitEvent(st, s.pool_free, 0));
        if (cs != st) AGNES_CHECK_HIP(hipStreamWaitEvent(st, b.needed, 0));
        if (b.prof) AGNES_CHECK_HIP(hipEventRecord(w.ev[2], st));
        AGNES_CHECK_HIP(hipMemcpyAsync(w.plan.ptr, w.plan_host.ptr, w.plan_used, hipMemcpyHostToDevice, st));
        const int32_t* plan = w.plan.as<int32_t>();
        const int64_t blk_bytes = s.rpb * s.row_bytes;
        ga.feat = s.pool.ptr;
        ga.tbuf = s.tbuf.as<int32_t>();
        ga.tch = tch;
        ga.pool_rows = (uint32_t)s.pool_rows;
        for (const TierRound& r : rounds) {
            if (r.n_upd)
                AGNES_LAUNCH(k_tbuf_update, dim3(grid_for(r.n_upd, 256)), dim3(kBlock), 0, st, plan + r.upd_at,
                                   r.n_upd, s.tbuf.as<int32_t>());
            if (r.n_miss) {
                // 32 workgroups keep the host link busy (about 50 GB/s, as with
                // 16384); while they wait on host reads, kernels of other
                // streams (later hyperbatches' sampling and needed-block
                // compaction) are starved, more so the more workgroups stage:
                // 512 leave a pipelined step at 18.9 ms, 64 at 13.8, 32 at 11.7;
                // 16 no longer saturate the link
                const int gs = std::min(r.n_miss, 32);
                if (blk_bytes % 16 == 0)
                    AGNES_LAUNCH(k_stage<u32x4>, dim3(gs), dim3(kBlock), 0, st, (const u32x4*)s.host_feat_dev,
                                       s.pool.as<u32x4>(), plan + r.miss_at, r.n_miss, blk_bytes / 16);
                else
                    AGNES_LAUNCH(k_stage<uint32_t>, dim3(gs), dim3(kBlock), 0, st,
                                       (const uint32_t*)s.host_feat_dev, s.pool.as<uint32_t>(), plan + r.miss_at,
                                       r.n_miss, blk_bytes / 4);
            }
            GatherArgs a = ga;
            a.base = r.e0;
            a.rows = r.e1 - r.e0;
            if (a.rows > 0) copy_rows(a);
        }
        if (cache) {
            // access counts, then admissions in ascending node order while the cache has room
            AGNES_LAUNCH(k_access_count, dim3(gl), dim3(kBlock), 0, st, rlk, tch, s.acc_count.as<uint32_t>(),
                               (uint32_t)std::min<int64_t>(s.cache_threshold, 0xFFFFFFFFll), flag, ctl);
            scan_counts(flag, off, &ctl->rows, rows, &ctl->tier_cand, part, st);
            const int ga2 = (int)std::max<int64_t>(1, std::min<int64_t>((rows + 3) / 4, 1 << 20));
            if (s.row_bytes % 16 == 0)
                AGNES_LAUNCH(k_admit<u32x4>, dim3(ga2), dim3(kBlock), 0, st, rlk, flag, off,
                                   (const u32x4*)s.host_feat_dev, s.pool.as<u32x4>(), s.pool_rows, s.row_bytes / 16,
                                   s.tch.as<int32_t>(), s.cache_used.as<int64_t>(), s.cache_rows, ctl);
            else
                AGNES_LAUNCH(k_admit<uint32_t>, dim3(ga2), dim3(kBlock), 0, st, rlk, flag, off,
                                   (const uint32_t*)s.host_feat_dev, s.pool.as<uint32_t>(), s.pool_rows,
                                   s.row_bytes / 4, s.tch.as<int32_t>(), s.cache_used.as<int64_t>(), s.cache_rows,
                                   ctl);
            AGNES_LAUNCH(k_admit_close, dim3(1), dim3(kWave), 0, st, s.cache_used.as<int64_t>(), s.cache_rows,
                               ctl);
        }
        AGNES_CHECK_HIP(hipGetLastError());
        // tier counters for wait
        AGNES_CHECK_HIP(hipMemcpyAsync(w.sync_host.ptr, ctl, sizeof(Ctl), hipMemcpyDeviceToHost, st));
        AGNES_CHECK_HIP(hipEventRecord(s.pool_free, st));
    } else {
        if (b.prof) AGNES_CHECK_HIP(hipEventRecord(w.ev[2], st));
        if (rows > 0) copy_rows(ga);
        AGNES_CHECK_HIP(hipGetLastError());
    }
    // the end of the gather (after the tier counters' copy): what wait waits for
    b.gathered_at = b.prof ? w.ev[4] : b.gathered;
    AGNES_CHECK_HIP(hipEventRecord(b.gathered_at, st));
    b.stream = st;
    b.state = kGathering;
}

void wait_batch(Batch& b) {
    if (b.state == kDone) return;
    Range range("agnes_batch_wait");
    AGNES_REQUIRE(b.state == kGathering, AGNES_ERR_INVALID, "the batch holds no finished hyperbatch");
    AGNES_CHECK_HIP(hipEventSynchronize(b.gathered_at));
    b.stats.sample_ms = b.stats.gather_ms = b.stats.copy_ms = -1.0f;
    if (b.prof) {
        Workspace& w = b.ws;
        AGNES_CHECK_HIP(hipEventElapsedTime(&b.stats.sample_ms, w.ev[0], w.ev[1]));
        AGNES_CHECK_HIP(hipEventElapsedTime(&b.stats.gather_ms, w.ev[2], w.ev[4]));
        b.stats.copy_ms = b.stats.gather_ms;
    }
    if (b.store->tiered) {
        b.tier.gather_ms = b.stats.gather_ms;
        if (b.node_off[b.H] > 0) {
            Ctl hc;
            memcpy(&hc, b.ws.sync_host.ptr, sizeof(Ctl));
            b.tier.cache_hit_rows = hc.tier_hits;
            b.tier.admitted_rows = hc.tier_admitted;
            b.tier.cached_rows = hc.tier_cached;
        }
    }
    b.state = kDone;
}

}  // namespace agnes
