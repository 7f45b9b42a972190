// The hyperbatch data-preparation pipeline (AGNES, arXiv 2601.01473, Alg. 1) on
// gfx950.
//
// Per hop l:
//   k_begin      per-minibatch bookkeeping: request offsets of the frontier
//   k_frontier   degree, k = min(deg, f_l), home topology block of every request
//                and the row sizes of the bucket matrix Bck (Sec. 3.4(3))
//   scans        edge offsets of the requests; Bck row offsets
//   k_bscatter   requests into their Bck rows (block-major order)
//   k_sample     Bck rows in block order: Floyd subsets from Philox words, the
//                sampled neighbours written at the request's edge offset, and the
//                hop's row pointers (Alg. 1, sampling loop)
//   k_insert     (minibatch, neighbour) into the hash table; first inserters are
//                the hop's new nodes (the union of Alg. 1)
//   scan         positions of the new nodes; k_compact gathers them
//   radix sort   new nodes by (minibatch, node id)
//   k_assign     local ids of the new nodes: |S_{l-1}| + rank
//   k_relabel    hop columns in local ids
// Gather (Alg. 1, gathering loop):
//   k_gkey       feature block of every output row, Bck row sizes, row bitmap
//   scan         Bck row offsets (and the number of non-empty rows)
//   k_gscatter   output rows into their Bck rows
//   k_gather     row copies in block order, 16-byte lanes, non-temporal stores
//
// All sizes produced on the device stay there until one synchronisation before
// the gather, where the host learns the output sizes.  Counters are combined
// per run of equal keys inside a wave (one atomic per run, all runs at once),
// and the new nodes are compacted with a scan rather than a shared counter.
#include <algorithm>
#include <cstring>

#include "device.hpp"
#include "runtime.hpp"

namespace agnes {

struct Geometry {
    int32_t H, B, L;
    int64_t capN;                      // node capacity of one minibatch
    int64_t cap[AGNES_MAX_LAYERS + 1]; // cap[l] = frontier capacity of hop l (cap[L] = capN)
    int64_t Rmax, Smax, rows_max;
    int jbits;
};

static Geometry plan(const Store& s, int32_t H, int32_t B, const int32_t* fanouts, int32_t L) {
    Geometry g{};
    g.H = H; g.B = B; g.L = L;
    int64_t c = std::min<int64_t>(B, s.num_nodes);
    if (B > s.num_nodes) c = B;        // duplicates are rejected later; keep room for them
    g.cap[0] = c;
    g.Rmax = 0; g.Smax = 0;
    for (int l = 0; l < L; l++) {
        g.Rmax = std::max<int64_t>(g.Rmax, (int64_t)H * g.cap[l]);
        g.Smax = std::max<int64_t>(g.Smax, (int64_t)H * g.cap[l] * fanouts[l]);
        int64_t nxt = g.cap[l] * (1 + (int64_t)fanouts[l]);
        nxt = std::min<int64_t>(nxt, std::max<int64_t>(s.num_nodes, g.cap[0]));
        g.cap[l + 1] = nxt;
    }
    g.capN = g.cap[L];
    g.rows_max = (int64_t)H * g.capN;
    int jb = 0;
    while ((1 << jb) < H) jb++;
    g.jbits = jb;
    return g;
}

// ----------------------------------------------------------------- kernels

// Load an int64 array of n+1 entries into shared memory.
__device__ __forceinline__ void load_offsets(int64_t* dst, const int64_t* src, int n) {
    for (int i = threadIdx.x; i <= n; i += kBlock) dst[i] = src[i];
    __syncthreads();
}

// Block 0: per-minibatch bookkeeping between hops.  Entering hop l (l < L) it
// closes hop l-1 (edge counts, node counts grown by the new nodes) and computes
// the request offsets of hop l; with l == L it closes the last hop and computes
// the output row offsets.  Other blocks clear the Bck row counters of hop l.
__global__ __launch_bounds__(kBlock) void k_begin(int l, int L, int H, Ctl* ctl, int32_t* size,
                                                  int64_t* newcnt, int32_t* lsz, int64_t* ecount,
                                                  int64_t* req_off, const int64_t* e_off,
                                                  int64_t* node_off, int64_t* bcnt, int64_t nblk) {
    if (blockIdx.x > 0) {
        if (l < L)
            for (int64_t i = (int64_t)(blockIdx.x - 1) * kBlock + threadIdx.x; i <= nblk;
                 i += (int64_t)(gridDim.x - 1) * kBlock)
                bcnt[i] = 0;
        return;
    }
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

// Reset the control block; the block counts are kept there for the scans.
__global__ void k_ctl_init(Ctl* ctl, int64_t nblk, int64_t nfblk) {
    int64_t* p = (int64_t*)ctl;
    for (int i = threadIdx.x; i < (int)(sizeof(Ctl) / 8); i += kBlock) p[i] = 0;
    __syncthreads();
    if (threadIdx.x == 0) {
        ctl->nblk = nblk;
        ctl->nfblk = nfblk;
    }
}

// Targets become the first B nodes of every minibatch.  An out-of-range target
// is recorded as an error and replaced by node 0 so that later kernels stay in
// bounds; a duplicate within a minibatch is recorded as an error.
__global__ __launch_bounds__(kBlock) void k_init(const int32_t* targets, int H, int B,
                                                 int64_t num_nodes, int node_bits, int64_t capN,
                                                 unsigned long long* ht_words, int32_t* ht_vals,
                                                 int ht_log2, int32_t* nodes, int32_t* size,
                                                 int64_t* newcnt, Ctl* ctl) {
    int64_t n = (int64_t)H * B;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += (int64_t)gridDim.x * kBlock) {
        int64_t j = i / B, r = i - j * B;
        int32_t v = targets[i];
        if (v < 0 || v >= num_nodes) {
            atomicOr((unsigned long long*)&ctl->err, 1ull);
            v = 0;
        } else {
            bool inserted, overflow;
            uint32_t slot = ht_insert(ht_words, ht_log2, ((uint64_t)j << node_bits) | (uint64_t)v, inserted,
                                      overflow);
            if (overflow) atomicOr((unsigned long long*)&ctl->err, 8ull);
            else if (inserted) ht_vals[slot] = (int32_t)r;
            else atomicOr((unsigned long long*)&ctl->err, 2ull);
        }
        nodes[j * capN + r] = v;
        if (r == 0) {
            size[j] = B;
            newcnt[j] = 0;
        }
    }
}

template <typename OffT>
__global__ __launch_bounds__(kBlock) void k_frontier(int H, int64_t capN, int32_t f,
                                                     const OffT* off, int e_blk_log2, int64_t nblk,
                                                     const int32_t* nodes, const int64_t* req_off_g,
                                                     int32_t* cnt, int32_t* bkey, int64_t* bcnt,
                                                     const Ctl* ctl) {
    extern __shared__ int64_t req_off[];
    load_offsets(req_off, req_off_g, H);
    const int64_t R = ctl->R;
    for (int64_t base = (int64_t)blockIdx.x * kBlock; base < R; base += (int64_t)gridDim.x * kBlock) {
        int64_t q = base + threadIdx.x;
        bool active = q < R;
        int64_t b = 0;
        if (active) {
            int j = upper_segment(req_off, H, q);
            int64_t r = q - req_off[j];
            int32_t v = nodes[(int64_t)j * capN + r];
            int64_t o0 = (int64_t)off[v], o1 = (int64_t)off[v + 1];
            int64_t deg = o1 - o0;
            cnt[q] = (int32_t)(deg < f ? deg : f);
            b = o0 >> e_blk_log2;
            if (b >= nblk) b = nblk - 1;
            bkey[q] = (int32_t)b;
        }
        run_count(bcnt, b, active);
    }
}

// Requests into their Bck rows: row b holds the requests whose home block is b.
__global__ __launch_bounds__(kBlock) void k_bscatter(const int32_t* bkey, int64_t* bcur,
                                                     int64_t* bck, const Ctl* ctl) {
    const int64_t R = ctl->R;
    for (int64_t base = (int64_t)blockIdx.x * kBlock; base < R; base += (int64_t)gridDim.x * kBlock) {
        int64_t q = base + threadIdx.x;
        bool active = q < R;
        int64_t key = active ? bkey[q] : 0;
        int64_t pos = run_increment(bcur, key, active);
        if (active) bck[pos] = q;
    }
}

// Sample every request, visiting the Bck rows in block order: consecutive
// threads serve requests of the same topology block, from every minibatch.
template <typename OffT, int MAXK>
__global__ __launch_bounds__(kBlock) void k_sample(int l, int H, int64_t capN, int32_t f,
                                                   uint64_t seed, int64_t mb_base, const OffT* off,
                                                   const int32_t* adj, const int32_t* nodes,
                                                   const int64_t* req_off_g, const int64_t* bck,
                                                   const int32_t* cnt, const int64_t* e_off,
                                                   int32_t* cg, int32_t* row_ptr, const Ctl* ctl) {
    extern __shared__ int64_t req_off[];
    load_offsets(req_off, req_off_g, H);
    const int64_t R = ctl->R;
    for (int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x; p < R; p += (int64_t)gridDim.x * kBlock) {
        int64_t q = bck[p];
        int j = upper_segment(req_off, H, q);
        int64_t r = q - req_off[j];
        int32_t v = nodes[(int64_t)j * capN + r];
        int64_t o0 = (int64_t)off[v];
        int64_t deg = (int64_t)off[v + 1] - o0;
        int k = cnt[q];
        int64_t eo = e_off[q];
        int64_t mb_e0 = e_off[req_off[j]];
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
}

// Union of Alg. 1: insert every sampled (minibatch, neighbour); the insert that
// creates a key marks a new node of the hop (flag[e] = 1).
__global__ __launch_bounds__(kBlock) void k_insert(int H, int node_bits, const int64_t* req_off_g,
                                                   const int64_t* e_off, const int32_t* cg,
                                                   unsigned long long* ht_words, int ht_log2,
                                                   uint32_t* eslot, int32_t* flag, Ctl* ctl) {
    extern __shared__ int64_t mb_e[];
    for (int i = threadIdx.x; i <= H; i += kBlock) mb_e[i] = e_off[req_off_g[i]];
    __syncthreads();
    const int64_t S = ctl->S;
    for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < S; e += (int64_t)gridDim.x * kBlock) {
        int j = upper_segment(mb_e, H, e);
        uint64_t key = ((uint64_t)j << node_bits) | (uint64_t)(uint32_t)cg[e];
        bool inserted, overflow;
        uint32_t slot = ht_insert(ht_words, ht_log2, key, inserted, overflow);
        if (overflow) atomicOr((unsigned long long*)&ctl->err, 8ull);
        eslot[e] = slot;
        flag[e] = inserted ? 1 : 0;
    }
}

// New node number fpre[e] of the hop: its sort key and hash slot.
__global__ __launch_bounds__(kBlock) void k_compact(int H, int node_bits, const int64_t* req_off_g,
                                                    const int64_t* e_off, const int32_t* cg,
                                                    const int32_t* flag, const int64_t* fpre,
                                                    const uint32_t* eslot, uint64_t* nkeys,
                                                    uint32_t* nvals, const Ctl* ctl) {
    extern __shared__ int64_t mb_e[];
    for (int i = threadIdx.x; i <= H; i += kBlock) mb_e[i] = e_off[req_off_g[i]];
    __syncthreads();
    const int64_t S = ctl->S;
    for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < S; e += (int64_t)gridDim.x * kBlock) {
        if (!flag[e]) continue;
        int j = upper_segment(mb_e, H, e);
        int64_t pos = fpre[e];
        nkeys[pos] = ((uint64_t)j << node_bits) | (uint64_t)(uint32_t)cg[e];
        nvals[pos] = eslot[e];
    }
}

// Per minibatch j: new nodes of the hop (newcnt) and
// base[j] = |S_{j,l-1}| - (start of minibatch j in the sorted new-node list).
__global__ __launch_bounds__(kBlock) void k_newbase(int H, const int32_t* size, const int64_t* req_off,
                                                    const int64_t* e_off, const int64_t* fpre,
                                                    int64_t* newcnt, int64_t* base) {
    for (int j = threadIdx.x; j < H; j += kBlock) {
        int64_t a = fpre[e_off[req_off[j]]], b = fpre[e_off[req_off[j + 1]]];
        newcnt[j] = b - a;
        base[j] = (int64_t)size[j] - a;
    }
}

// New nodes in (minibatch, id) order get local ids |S_{j,l-1}| + rank.
__global__ __launch_bounds__(kBlock) void k_assign(int H, int node_bits, int64_t capN,
                                                   const uint64_t* nkeys, const uint32_t* nvals,
                                                   const int64_t* base_g, int32_t* ht_vals,
                                                   int32_t* nodes, Ctl* ctl) {
    extern __shared__ int64_t base[];
    for (int i = threadIdx.x; i < H; i += kBlock) base[i] = base_g[i];
    __syncthreads();
    const int64_t n = ctl->n_new;
    const uint64_t umask = (1ull << node_bits) - 1;
    for (int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x; p < n; p += (int64_t)gridDim.x * kBlock) {
        uint64_t key = nkeys[p];
        int j = (int)(key >> node_bits);
        int64_t local = base[j] + p;
        if (local >= capN || local >= 0x7FFFFFFF) {
            atomicOr((unsigned long long*)&ctl->err, 4ull);
            continue;
        }
        ht_vals[nvals[p]] = (int32_t)local;
        nodes[(int64_t)j * capN + local] = (int32_t)(key & umask);
    }
}

__global__ __launch_bounds__(kBlock) void k_relabel(const uint32_t* eslot, const int32_t* ht_vals,
                                                    int32_t* col, const Ctl* ctl) {
    const int64_t S = ctl->S;
    for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < S; e += (int64_t)gridDim.x * kBlock)
        col[e] = ht_vals[eslot[e]];
}

// ----------------------------------------------------------------- gather kernels

// Output row i of minibatch j is node nodes[j][i - node_off[j]]; its feature
// block is the Bck row it falls in.  dbits marks every gathered node.
__global__ __launch_bounds__(kBlock) void k_gkey(int H, int64_t capN, const int64_t* node_off_g,
                                                 const int32_t* nodes, int32_t* nodes_out,
                                                 int32_t rpb, int32_t* gkey, int64_t* fbcnt,
                                                 uint32_t* dbits, const Ctl* ctl) {
    extern __shared__ int64_t node_off[];
    load_offsets(node_off, node_off_g, H);
    const int64_t rows = ctl->rows;
    for (int64_t base = (int64_t)blockIdx.x * kBlock; base < rows; base += (int64_t)gridDim.x * kBlock) {
        int64_t i = base + threadIdx.x;
        bool active = i < rows;
        int64_t fb = 0;
        if (active) {
            int j = upper_segment(node_off, H, i);
            int32_t v = nodes[(int64_t)j * capN + (i - node_off[j])];
            nodes_out[i] = v;
            fb = (uint32_t)v / (uint32_t)rpb;
            gkey[i] = (int32_t)fb;
            atomicOr(&dbits[v >> 5], 1u << (v & 31));
        }
        run_count(fbcnt, fb, active);
    }
}

// Number of set bits of a bitmap, added to *out.
__global__ __launch_bounds__(kBlock) void k_popcount(const uint32_t* bits, int64_t nwords, int64_t* out) {
    __shared__ int64_t lds[kWavesPerBlock];
    int64_t c = 0;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < nwords; i += (int64_t)gridDim.x * kBlock)
        c += __popc(bits[i]);
    c = wave_inclusive_scan(c);
    if (lane_id() == kWave - 1) lds[wave_id()] = c;
    __syncthreads();
    if (threadIdx.x == 0) {
        int64_t t = 0;
        for (int w = 0; w < kWavesPerBlock; w++) t += lds[w];
        if (t) atomicAdd((unsigned long long*)out, (unsigned long long)t);
    }
}

__global__ __launch_bounds__(kBlock) void k_gscatter(const int32_t* gkey, const int32_t* nodes_out,
                                                     int64_t* fbcur, uint64_t* gent, const Ctl* ctl) {
    const int64_t rows = ctl->rows;
    for (int64_t base = (int64_t)blockIdx.x * kBlock; base < rows; base += (int64_t)gridDim.x * kBlock) {
        int64_t i = base + threadIdx.x;
        bool active = i < rows;
        int64_t key = active ? gkey[i] : 0;
        int64_t pos = run_increment(fbcur, key, active);
        if (active) gent[pos] = ((uint64_t)i << 32) | (uint32_t)nodes_out[i];
    }
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Row copy in Bck order.  LPR lanes share a row (Unit = 16 or 4 bytes per lane
// access), each group moves two rows per step so that two loads are in flight
// before the stores.  Workgroup b processes a contiguous range of entries; the
// ranges are assigned so that neighbouring ranges (the same feature blocks) run
// on the same XCD (workgroups are dealt to the 8 XCDs round-robin).
template <typename Unit, int LPR>
__global__ __launch_bounds__(kBlock) void k_gather(const Unit* __restrict__ feat, Unit* __restrict__ out,
                                                   const uint64_t* __restrict__ gent, int64_t rows,
                                                   int64_t row_units) {
    constexpr int RPW = kWave / LPR;             // rows per wave access
    const int G = gridDim.x;
    const int b = blockIdx.x;
    const int lb = (G % 8 == 0) ? (b % 8) * (G / 8) + b / 8 : b;
    const int64_t chunk = (rows + G - 1) / G;
    const int64_t lo = std::min<int64_t>(rows, (int64_t)lb * chunk);
    const int64_t hi = std::min<int64_t>(rows, lo + chunk);
    const int grp = lane_id() / LPR, li = lane_id() % LPR;
    const int64_t step = (int64_t)kWavesPerBlock * RPW;
    for (int64_t e = lo + (int64_t)wave_id() * RPW + grp; e < hi; e += 2 * step) {
        int64_t e2 = e + step;
        uint64_t ga = gent[e];
        uint64_t gb = (e2 < hi) ? gent[e2] : 0;
        const Unit* sa = feat + (int64_t)(uint32_t)ga * row_units;
        const Unit* sb = feat + (int64_t)(uint32_t)gb * row_units;
        Unit* da = out + (int64_t)(ga >> 32) * row_units;
        Unit* db = out + (int64_t)(gb >> 32) * row_units;
        for (int64_t u = li; u < row_units; u += LPR) {
            Unit xa = sa[u];
            Unit xb;
            if (e2 < hi) xb = sb[u];
            __builtin_nontemporal_store(xa, da + u);
            if (e2 < hi) __builtin_nontemporal_store(xb, db + u);
        }
    }
}

template <typename Unit>
static void launch_gather(const void* feat, void* out, const uint64_t* gent, int64_t rows,
                          int64_t row_units, hipStream_t st) {
    int G = grid_for(rows * row_units / 64 + 1, 8192);
    G = std::max(8, (G + 7) / 8 * 8);
    const Unit* f = (const Unit*)feat;
    Unit* o = (Unit*)out;
    if (row_units >= 64)
        hipLaunchKernelGGL((k_gather<Unit, 64>), dim3(G), dim3(kBlock), 0, st, f, o, gent, rows, row_units);
    else if (row_units > 16)
        hipLaunchKernelGGL((k_gather<Unit, 32>), dim3(G), dim3(kBlock), 0, st, f, o, gent, rows, row_units);
    else if (row_units > 8)
        hipLaunchKernelGGL((k_gather<Unit, 16>), dim3(G), dim3(kBlock), 0, st, f, o, gent, rows, row_units);
    else if (row_units > 4)
        hipLaunchKernelGGL((k_gather<Unit, 8>), dim3(G), dim3(kBlock), 0, st, f, o, gent, rows, row_units);
    else
        hipLaunchKernelGGL((k_gather<Unit, 4>), dim3(G), dim3(kBlock), 0, st, f, o, gent, rows, row_units);
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

template <typename OffT>
static void launch_layer(Store& s, const Geometry& g, int l, int32_t f, uint64_t seed, int64_t mb_base,
                         Batch& b, const SyncLayout& y, hipStream_t st) {
    Workspace& w = s.ws;
    Ctl* ctl = w.sync.as<Ctl>();
    int32_t* lsz = (int32_t*)((char*)w.sync.ptr + y.lsz);
    int64_t* ecount = (int64_t*)((char*)w.sync.ptr + y.ecount);
    const OffT* off = s.offsets.as<OffT>();
    const size_t lds_req = (size_t)(g.H + 1) * sizeof(int64_t);
    const int gR = grid_for(g.Rmax, 2048);
    const int gS = grid_for(g.Smax, 4096);
    int64_t* part = w.scan_part.as<int64_t>();

    hipLaunchKernelGGL(k_begin, dim3(1 + grid_for(s.nblk + 1, 256)), dim3(kBlock), 0, st, l, g.L, g.H, ctl,
                       w.size.as<int32_t>(), w.newcnt.as<int64_t>(), lsz, ecount, w.req_off.as<int64_t>(),
                       w.e_off.as<int64_t>(), (int64_t*)nullptr, w.bcnt.as<int64_t>(), s.nblk);
    hipLaunchKernelGGL(k_frontier<OffT>, dim3(gR), dim3(kBlock), lds_req, st, g.H, g.capN, f, off,
                       s.e_blk_log2, s.nblk, w.nodes.as<int32_t>(), w.req_off.as<int64_t>(),
                       w.cnt.as<int32_t>(), w.bkey.as<int32_t>(), w.bcnt.as<int64_t>(), ctl);
    scan_counts(w.cnt.as<int32_t>(), w.e_off.as<int64_t>(), &ctl->R, g.Rmax, &ctl->S, part, st);
    // Bck row offsets over the topology blocks; the non-empty rows are T_l
    scan_counts64(w.bcnt.as<int64_t>(), w.bcur.as<int64_t>(), &ctl->nblk, s.nblk, nullptr, part, st,
                  &ctl->topo_blocks[l]);
    hipLaunchKernelGGL(k_bscatter, dim3(gR), dim3(kBlock), 0, st, w.bkey.as<int32_t>(),
                       w.bcur.as<int64_t>(), w.bck.as<int64_t>(), ctl);
    int32_t* rp = b.row_ptr[l].as<int32_t>();
    const int32_t* adj = s.indices.as<int32_t>();
#define AGNES_SAMPLE(MK)                                                                          \
    hipLaunchKernelGGL((k_sample<OffT, MK>), dim3(gR), dim3(kBlock), lds_req, st, l, g.H, g.capN, f,\
                       seed, mb_base, off, adj, w.nodes.as<int32_t>(), w.req_off.as<int64_t>(),   \
                       w.bck.as<int64_t>(), w.cnt.as<int32_t>(), w.e_off.as<int64_t>(),           \
                       w.cg.as<int32_t>(), rp, ctl)
    if (f <= 4) AGNES_SAMPLE(4);
    else if (f <= 8) AGNES_SAMPLE(8);
    else if (f <= 16) AGNES_SAMPLE(16);
    else if (f <= 32) AGNES_SAMPLE(32);
    else AGNES_SAMPLE(0);
#undef AGNES_SAMPLE
    hipLaunchKernelGGL(k_insert, dim3(gS), dim3(kBlock), lds_req, st, g.H, s.node_bits,
                       w.req_off.as<int64_t>(), w.e_off.as<int64_t>(), w.cg.as<int32_t>(),
                       w.ht_words.as<unsigned long long>(), w.ht_log2, w.eslot.as<uint32_t>(),
                       w.flag.as<int32_t>(), ctl);
    scan_counts(w.flag.as<int32_t>(), w.fpre.as<int64_t>(), &ctl->S, g.Smax, &ctl->n_new, part, st);
    hipLaunchKernelGGL(k_compact, dim3(gS), dim3(kBlock), lds_req, st, g.H, s.node_bits,
                       w.req_off.as<int64_t>(), w.e_off.as<int64_t>(), w.cg.as<int32_t>(),
                       w.flag.as<int32_t>(), w.fpre.as<int64_t>(), w.eslot.as<uint32_t>(),
                       w.nkeys.as<uint64_t>(), w.nvals.as<uint32_t>(), ctl);
    int in_tmp = radix_sort_pairs(w.nkeys.as<uint64_t>(), w.nvals.as<uint32_t>(), w.nkeys2.as<uint64_t>(),
                                  w.nvals2.as<uint32_t>(), &ctl->n_new, g.Smax, s.node_bits + g.jbits,
                                  w.rs_hist.as<int64_t>(), w.rs_dtot.as<int64_t>(), st);
    const uint64_t* skeys = in_tmp ? w.nkeys2.as<uint64_t>() : w.nkeys.as<uint64_t>();
    const uint32_t* svals = in_tmp ? w.nvals2.as<uint32_t>() : w.nvals.as<uint32_t>();
    hipLaunchKernelGGL(k_newbase, dim3(1), dim3(kBlock), 0, st, g.H, w.size.as<int32_t>(),
                       w.req_off.as<int64_t>(), w.e_off.as<int64_t>(), w.fpre.as<int64_t>(),
                       w.newcnt.as<int64_t>(), w.mb_off.as<int64_t>());
    hipLaunchKernelGGL(k_assign, dim3(gS), dim3(kBlock), (size_t)g.H * sizeof(int64_t), st, g.H,
                       s.node_bits, g.capN, skeys, svals, w.mb_off.as<int64_t>(), w.ht_vals.as<int32_t>(),
                       w.nodes.as<int32_t>(), ctl);
    hipLaunchKernelGGL(k_relabel, dim3(gS), dim3(kBlock), 0, st, w.eslot.as<uint32_t>(),
                       w.ht_vals.as<int32_t>(), b.col[l].as<int32_t>(), ctl);
    AGNES_CHECK_HIP(hipGetLastError());
}

static int ceil_log2(int64_t x) {
    int lg = 0;
    while (((int64_t)1 << lg) < x) lg++;
    return lg;
}

static void reserve_workspace(Store& s, const Geometry& g, const SyncLayout& y) {
    Workspace& w = s.ws;
    const int64_t H = g.H;
    // hash table: one key per (minibatch, node); at most half full in the worst
    // case, about a third full when sized from the rows seen so far
    int lg_max = std::max(10, ceil_log2(2 * g.rows_max));
    int lg = s.ht_hint > 0 ? std::max(10, ceil_log2(3 * s.ht_hint)) : lg_max;
    lg = std::min(std::max(lg, s.ht_min_log2), lg_max);
    AGNES_REQUIRE(lg <= 31, AGNES_ERR_RANGE, "hyperbatch too large for the 2^31-slot hash table");
    w.ht_log2 = lg;
    w.ht_words.reserve(((size_t)1 << lg) * 8);
    w.ht_vals.reserve(((size_t)1 << lg) * 4);
    w.nodes.reserve((size_t)g.rows_max * 4);
    w.size.reserve((size_t)H * 4);
    w.newcnt.reserve((size_t)H * 8);
    w.req_off.reserve((size_t)(H + 1) * 8);
    w.mb_off.reserve((size_t)(H + 1) * 8);
    w.sync.reserve(y.bytes);
    w.sync_host.reserve(y.bytes);
    w.cnt.reserve((size_t)g.Rmax * 4);
    w.bkey.reserve((size_t)g.Rmax * 4);
    w.bck.reserve((size_t)g.Rmax * 8);
    w.e_off.reserve((size_t)(g.Rmax + 1) * 8);
    w.bcnt.reserve((size_t)(s.nblk + 1) * 8);
    w.bcur.reserve((size_t)(s.nblk + 2) * 8);
    w.cg.reserve((size_t)g.Smax * 4);
    w.eslot.reserve((size_t)g.Smax * 4);
    w.flag.reserve((size_t)g.Smax * 4);
    w.fpre.reserve((size_t)(g.Smax + 1) * 8);
    w.nkeys.reserve((size_t)g.Smax * 8);
    w.nkeys2.reserve((size_t)g.Smax * 8);
    w.nvals.reserve((size_t)g.Smax * 4);
    w.nvals2.reserve((size_t)g.Smax * 4);
    w.rs_hist.reserve((size_t)radix_hist_entries() * 8);
    w.rs_dtot.reserve((size_t)radix_dtot_entries() * 8);
    w.scan_part.reserve((size_t)scan_partials_needed() * 8);
    w.gkey.reserve((size_t)g.rows_max * 4);
    w.gent.reserve((size_t)g.rows_max * 8);
    w.fbcnt.reserve((size_t)(s.nfblk + 1) * 8);
    w.fbcur.reserve((size_t)(s.nfblk + 2) * 8);
    w.dbits.reserve((size_t)((s.num_nodes + 31) / 32) * 4);
    if (!w.ev[0])
        for (auto& e : w.ev) AGNES_CHECK_HIP(hipEventCreate(&e));
}

// Sampling of all hops; returns false when the hash table overflowed (the host
// then grows it and runs again).
static bool run_sampling(Store& s, Batch& b, const Geometry& g, const SyncLayout& y,
                         const int32_t* targets, const int32_t* fanouts, uint64_t seed,
                         int64_t mb_base, hipStream_t st, Ctl& hc, std::vector<int64_t>& ecount) {
    Workspace& w = s.ws;
    reserve_workspace(s, g, y);
    Ctl* ctl = w.sync.as<Ctl>();
    int32_t* lsz = (int32_t*)((char*)w.sync.ptr + y.lsz);
    int64_t* ec = (int64_t*)((char*)w.sync.ptr + y.ecount);
    const int H = g.H, B = g.B, L = g.L;

    if (s.profile) AGNES_CHECK_HIP(hipEventRecord(w.ev[0], st));
    hipLaunchKernelGGL(k_ctl_init, dim3(1), dim3(kBlock), 0, st, ctl, s.nblk, s.nfblk);
    fill_u32(w.ht_words.ptr, 0, ((int64_t)1 << w.ht_log2) * 2, st);
    hipLaunchKernelGGL(k_init, dim3(grid_for((int64_t)H * B, 1024)), dim3(kBlock), 0, st, targets, H, B,
                       s.num_nodes, s.node_bits, g.capN, w.ht_words.as<unsigned long long>(),
                       w.ht_vals.as<int32_t>(), w.ht_log2, w.nodes.as<int32_t>(), w.size.as<int32_t>(),
                       w.newcnt.as<int64_t>(), ctl);
    AGNES_CHECK_HIP(hipGetLastError());
    for (int l = 0; l < L; l++) {
        if (s.offsets64) launch_layer<int64_t>(s, g, l, fanouts[l], seed, mb_base, b, y, st);
        else launch_layer<int32_t>(s, g, l, fanouts[l], seed, mb_base, b, y, st);
    }
    // close the last hop: edge counts, final node counts, output row offsets
    hipLaunchKernelGGL(k_begin, dim3(1), dim3(kBlock), 0, st, L, L, H, ctl, w.size.as<int32_t>(),
                       w.newcnt.as<int64_t>(), lsz, ec, w.req_off.as<int64_t>(), w.e_off.as<int64_t>(),
                       w.mb_off.as<int64_t>(), w.bcnt.as<int64_t>(), s.nblk);
    AGNES_CHECK_HIP(hipGetLastError());
    if (s.profile) AGNES_CHECK_HIP(hipEventRecord(w.ev[1], st));

    // the one host synchronisation: sizes of the outputs
    AGNES_CHECK_HIP(hipMemcpyAsync(w.sync_host.ptr, w.sync.ptr, y.bytes, hipMemcpyDeviceToHost, st));
    AGNES_CHECK_HIP(hipStreamSynchronize(st));
    memcpy(&hc, w.sync_host.ptr, sizeof(Ctl));
    b.layer_sizes.assign((size_t)H * (L + 1), 0);
    memcpy(b.layer_sizes.data(), (char*)w.sync_host.ptr + y.lsz, b.layer_sizes.size() * 4);
    ecount.assign((size_t)H * L, 0);
    memcpy(ecount.data(), (char*)w.sync_host.ptr + y.ecount, ecount.size() * 8);
    return !(hc.err & 8);
}

void prepare_hyperbatch(Store& s, Batch& b, const int32_t* targets, int32_t H, int32_t B,
                        const int32_t* fanouts, int32_t L, uint64_t seed, int64_t mb_base,
                        hipStream_t st) {
    Geometry g = plan(s, H, B, fanouts, L);
    SyncLayout y = sync_layout(H, L);
    Workspace& w = s.ws;

    // outputs with worst-case capacity for the per-hop CSR
    b.store = &s;
    b.H = H; b.B = B; b.L = L;
    for (int l = 0; l < L; l++) {
        b.row_ptr[l].reserve((size_t)(H * g.cap[l] + H) * 4);
        b.col[l].reserve((size_t)std::max<int64_t>(1, H * g.cap[l] * fanouts[l]) * 4);
    }

    Ctl hc{};
    std::vector<int64_t> ecount;
    while (!run_sampling(s, b, g, y, targets, fanouts, seed, mb_base, st, hc, ecount)) {
        // the table was sized from earlier hyperbatches and this one did not fit
        AGNES_REQUIRE(w.ht_log2 < std::max(10, ceil_log2(2 * g.rows_max)), AGNES_ERR_INTERNAL,
                      "hash table overflow at its worst-case size");
        s.ht_min_log2 = w.ht_log2 + 1;
    }
    Ctl* ctl = w.sync.as<Ctl>();
    AGNES_REQUIRE(!(hc.err & 1), AGNES_ERR_INVALID, "a target is outside [0, num_nodes)");
    AGNES_REQUIRE(!(hc.err & 2), AGNES_ERR_INVALID, "a target appears twice in one minibatch");
    AGNES_REQUIRE(!(hc.err & 4), AGNES_ERR_INTERNAL, "node capacity exceeded");

    // host view offsets
    b.node_off.assign((size_t)H + 1, 0);
    for (int j = 0; j < H; j++) {
        int64_t n = b.layer_sizes[(size_t)j * (L + 1) + L];
        b.node_off[j + 1] = b.node_off[j] + n;
    }
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
    s.ht_hint = std::max<int64_t>(s.ht_hint, rows);
    b.nodes.reserve_slack((size_t)std::max<int64_t>(rows, 1) * 4);
    b.features.reserve_slack((size_t)std::max<int64_t>(rows, 1) * (size_t)s.row_bytes);

    // gather
    if (s.profile) AGNES_CHECK_HIP(hipEventRecord(w.ev[2], st));
    fill_u32(w.fbcnt.ptr, 0, (s.nfblk + 1) * 2, st);
    const int64_t nwords = (s.num_nodes + 31) / 32;
    fill_u32(w.dbits.ptr, 0, nwords, st);
    const size_t lds_node = (size_t)(H + 1) * sizeof(int64_t);
    const int gG = grid_for(rows, 4096);
    hipLaunchKernelGGL(k_gkey, dim3(gG), dim3(kBlock), lds_node, st, H, g.capN, w.mb_off.as<int64_t>(),
                       w.nodes.as<int32_t>(), b.nodes.as<int32_t>(), (int32_t)s.rpb, w.gkey.as<int32_t>(),
                       w.fbcnt.as<int64_t>(), w.dbits.as<uint32_t>(), ctl);
    hipLaunchKernelGGL(k_popcount, dim3(grid_for(nwords, 1024)), dim3(kBlock), 0, st, w.dbits.as<uint32_t>(),
                       nwords, &ctl->distinct);
    scan_counts64(w.fbcnt.as<int64_t>(), w.fbcur.as<int64_t>(), &ctl->nfblk, s.nfblk, nullptr,
                  w.scan_part.as<int64_t>(), st, &ctl->fblocks);
    hipLaunchKernelGGL(k_gscatter, dim3(gG), dim3(kBlock), 0, st, w.gkey.as<int32_t>(), b.nodes.as<int32_t>(),
                       w.fbcur.as<int64_t>(), w.gent.as<uint64_t>(), ctl);
    if (s.profile) AGNES_CHECK_HIP(hipEventRecord(w.ev[3], st));
    if (rows > 0) {
        if (s.row_bytes % 16 == 0)
            launch_gather<u32x4>(s.features.ptr, b.features.ptr, w.gent.as<uint64_t>(), rows, s.row_bytes / 16, st);
        else
            launch_gather<uint32_t>(s.features.ptr, b.features.ptr, w.gent.as<uint64_t>(), rows, s.row_bytes / 4, st);
    }
    AGNES_CHECK_HIP(hipGetLastError());
    if (s.profile) AGNES_CHECK_HIP(hipEventRecord(w.ev[4], st));
    AGNES_CHECK_HIP(hipMemcpyAsync(w.sync_host.ptr, ctl, sizeof(Ctl), hipMemcpyDeviceToHost, st));
    AGNES_CHECK_HIP(hipStreamSynchronize(st));
    memcpy(&hc, w.sync_host.ptr, sizeof(Ctl));

    // statistics
    agnes_stats& so = b.stats;
    memset(&so, 0, sizeof(so));
    so.L = L;
    for (int l = 0; l < L; l++) {
        so.requests[l] = hc.requests[l];
        so.sampled[l] = hc.sampled[l];
        so.new_nodes[l] = hc.new_nodes[l];
        so.topo_blocks[l] = hc.topo_blocks[l];
    }
    so.rows = rows;
    so.distinct_rows = hc.distinct;
    so.feat_blocks = hc.fblocks;
    so.sample_ms = so.gather_ms = so.copy_ms = -1.0f;
    if (s.profile) {
        AGNES_CHECK_HIP(hipEventElapsedTime(&so.sample_ms, w.ev[0], w.ev[1]));
        AGNES_CHECK_HIP(hipEventElapsedTime(&so.gather_ms, w.ev[2], w.ev[4]));
        AGNES_CHECK_HIP(hipEventElapsedTime(&so.copy_ms, w.ev[3], w.ev[4]));
    }
}

}  // namespace agnes
