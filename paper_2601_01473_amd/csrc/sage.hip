// GraphSAGE forward over a prepared hyperbatch (Eq. (1), Sec. 3.1): the
// computation step that consumes the per-hop CSR blocks and gathered rows.
//
// Layer i runs on hop l = L-1-i.  Per layer two kernels:
//   k_sage_agg   one lane group per destination node: its own input row and
//                the float32 mean of its sampled neighbours' rows, both rounded
//                to bf16, as one row [h_v ; m_v] of A (M x 2d, row-major);
//   k_sage_gemm  Z = A W^T + b with bf16 MFMA (32x32x16, float32 accumulate),
//                ReLU on hidden layers; hidden outputs stored as bf16, the last
//                layer's as float32.
// Destination rows of all minibatches are stacked minibatch-major, so a layer
// is one GEMM over the whole hyperbatch.
#include <algorithm>
#include <cstring>
#include <mutex>
#include <string>
#include <type_traits>
#include <vector>

#include "device.hpp"
#include "runtime.hpp"

namespace agnes {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));
typedef unsigned int u32x4s __attribute__((ext_vector_type(4)));

// float -> bf16 bits, round to nearest, ties to even (finite inputs).
__device__ __forceinline__ uint16_t to_bf16(float x) {
    uint32_t u = __float_as_uint(x);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float bf16_to_float(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// Sixteen bytes of consecutive input elements (4 float or 8 half / bf16) as float.
template <typename InT> struct In16;
template <> struct In16<float> {
    static constexpr int E = 4;
    static __device__ __forceinline__ void load(const float* p, float (&x)[E]) {
        const f32x4 v = *(const f32x4*)p;
        x[0] = v.x; x[1] = v.y; x[2] = v.z; x[3] = v.w;
    }
};
template <> struct In16<_Float16> {
    static constexpr int E = 8;
    static __device__ __forceinline__ void load(const _Float16* p, float (&x)[E]) {
        typedef _Float16 h8 __attribute__((ext_vector_type(8)));
        const h8 v = *(const h8*)p;
#pragma unroll
        for (int q = 0; q < E; q++) x[q] = (float)v[q];
    }
};
template <> struct In16<uint16_t> {   // bf16 bits
    static constexpr int E = 8;
    static __device__ __forceinline__ void load(const uint16_t* p, float (&x)[E]) {
        const u16x8 v = *(const u16x8*)p;
#pragma unroll
        for (int q = 0; q < E; q++) x[q] = bf16_to_float(v[q]);
    }
};

// E bf16 values (E = 4 or 8) as one 8- or 16-byte store.
template <int E> __device__ __forceinline__ void store_bf16(uint16_t* p, const float (&x)[E]);
template <> __device__ __forceinline__ void store_bf16<4>(uint16_t* p, const float (&x)[4]) {
    *(u16x4*)p = u16x4{to_bf16(x[0]), to_bf16(x[1]), to_bf16(x[2]), to_bf16(x[3])};
}
template <> __device__ __forceinline__ void store_bf16<8>(uint16_t* p, const float (&x)[8]) {
    u16x8 v;
#pragma unroll
    for (int q = 0; q < 8; q++) v[q] = to_bf16(x[q]);
    *(u16x8*)p = v;
}

// Offsets of one layer, all [H+1] int64: destination rows of minibatch j are
// [d_off[j], d_off[j+1]); its input rows start at in_off[j]; its hop-l row
// pointers at rp_off[j] and columns at col_off[j].
struct LayerOffsets {
    const int64_t* d_off;
    const int64_t* in_off;
    const int64_t* rp_off;
    const int64_t* col_off;
};

// One group of LPR lanes per destination row (64 / LPR rows per wave), each
// lane holding 16 bytes of the row per chunk: LPR = 64 for rows of 1 KiB and
// up, fewer lanes for narrower rows so that no lane idles.
template <typename InT, int LPR>
__global__ __launch_bounds__(kBlock) void k_sage_agg(const InT* __restrict__ hin, LayerOffsets o,
                                                     const int32_t* __restrict__ row_ptr,
                                                     const int32_t* __restrict__ col, int H, int64_t M, int din,
                                                     uint16_t* __restrict__ A) {
    constexpr int E = In16<InT>::E, RPW = kWave / LPR;
    const int lane = lane_id();
    const int g = RPW == 1 ? 0 : lane / LPR;        // a whole wave per row keeps the row's indices uniform
    const int gl = RPW == 1 ? lane : lane % LPR;
    const int64_t nw = (int64_t)gridDim.x * kWavesPerBlock;
    for (int64_t r0 = ((int64_t)blockIdx.x * kWavesPerBlock + wave_id()) * RPW; r0 < M; r0 += nw * RPW) {
        const int64_t row = r0 + g;
        if (row >= M) break;
        const int j = upper_segment(o.d_off, H, row);
        const int64_t v = row - o.d_off[j];
        const int32_t* rp = row_ptr + o.rp_off[j] + v;
        const int32_t beg = rp[0], end = rp[1];
        const int32_t* cb = col + o.col_off[j];
        const InT* base = hin + o.in_off[j] * (int64_t)din;
        uint16_t* arow = A + row * 2 * (int64_t)din;
        for (int c = gl * E; c < din; c += LPR * E) {
            float self[E], acc[E];
            In16<InT>::load(base + v * din + c, self);
#pragma unroll
            for (int q = 0; q < E; q++) acc[q] = 0.f;
            int32_t t = beg;
            for (; t + 4 <= end; t += 4) {
                const int32_t u0 = cb[t], u1 = cb[t + 1], u2 = cb[t + 2], u3 = cb[t + 3];
                float x0[E], x1[E], x2[E], x3[E];
                In16<InT>::load(base + (int64_t)u0 * din + c, x0);
                In16<InT>::load(base + (int64_t)u1 * din + c, x1);
                In16<InT>::load(base + (int64_t)u2 * din + c, x2);
                In16<InT>::load(base + (int64_t)u3 * din + c, x3);
#pragma unroll
                for (int q = 0; q < E; q++) acc[q] = (((acc[q] + x0[q]) + x1[q]) + x2[q]) + x3[q];
            }
            for (; t < end; t++) {
                float x[E];
                In16<InT>::load(base + (int64_t)cb[t] * din + c, x);
#pragma unroll
                for (int q = 0; q < E; q++) acc[q] += x[q];
            }
            const int deg = end - beg;
            if (deg > 0) {
                const float d = (float)deg;
#pragma unroll
                for (int q = 0; q < E; q++) acc[q] = acc[q] / d;
            }
            store_bf16<E>(arow + c, self);
            store_bf16<E>(arow + din + c, acc);
        }
    }
}

// Z[M][N] = A[M][K] W[N][K]^T + b.  Workgroup tile 128 x 128, K step 64; wave
// w owns the 64 x 64 quarter (w / 2, w % 2) as 2 x 2 MFMA 32x32 blocks.
// Operand layout of v_mfma_f32_32x32x16_bf16 (the CDNA4 instruction with twice
// the K depth of the 32x32x8 one at the same cycle count): lane l holds
// X[l % 32][8 (l / 32) + q] of the first operand and Y[8 (l / 32) + q][l % 32]
// of the second for q = 0..7, and D[8 (r / 4) + 4 (l / 32) + r % 4][l % 32] for
// r = 0..15.  W is stored output-major, so both tiles sit in LDS with k
// innermost and every operand is one 16-byte LDS read.  W's rows go in as the
// first operand and A's as the second, so D is a block of Z^T: lane l holds
// row l % 32 of Z and four adjacent columns per group of four registers.  The
// next K step's tiles are loaded into registers while the MFMAs consume the
// current ones.
constexpr int kGM = 128, kGN = 128, kGK = 64, kGKP = kGK + 8;   // padded LDS row (uint16)
constexpr int kGLoads = kGM * kGK / 8 / kBlock;                 // 16-byte pieces per thread per tile (4)

template <bool RELU, bool OUT_F32>
__global__ __launch_bounds__(kBlock) void k_sage_gemm(const uint16_t* __restrict__ A, const uint16_t* __restrict__ W,
                                                      const float* __restrict__ bias, int64_t M, int N, int K,
                                                      void* __restrict__ Z) {
    // one LDS block: the operand tiles during the K loop, the output tile after it
    __shared__ __attribute__((aligned(16))) uint16_t smem[(kGM + kGN) * kGKP];
    uint16_t (*As)[kGKP] = reinterpret_cast<uint16_t (*)[kGKP]>(smem);
    uint16_t (*Bs)[kGKP] = reinterpret_cast<uint16_t (*)[kGKP]>(smem + kGM * kGKP);
    const int lane = lane_id(), w = wave_id(), t = threadIdx.x;
    // Tile of workgroup i (1-D grid): runs of 8 NB workgroups cover 8 row
    // blocks x NB column blocks.  Workgroups i and i + 8 share an XCD (they are
    // dealt to the 8 XCDs in turn) and follow each other there, so the column
    // blocks of one row block run back to back on one XCD and all but the
    // first read its A tile from that XCD's L2.
    const int NB = (N + kGN - 1) / kGN;
    const int64_t i = blockIdx.x;
    const int64_t mb = (i / (8 * (int64_t)NB)) * 8 + (i % 8);
    const int64_t m0 = mb * kGM;
    const int n0 = (int)((i / 8) % NB) * kGN;
    if (m0 >= M) return;
    const int wm = (w >> 1) * 64, wn = (w & 1) * 64;
    f32x16 acc[2][2];
#pragma unroll
    for (int a = 0; a < 2; a++)
#pragma unroll
        for (int b = 0; b < 2; b++)
#pragma unroll
            for (int r = 0; r < 16; r++) acc[a][b][r] = 0.f;
    // piece p of thread t: row (t + p * 256) / 8, k offset ((t + p * 256) % 8) * 8
    u32x4s ra[kGLoads], rb[kGLoads];
    auto fetch = [&](int k0) {
#pragma unroll
        for (int p = 0; p < kGLoads; p++) {
            const int idx = t + p * kBlock;
            const int r = idx >> 3, kk = (idx & 7) * 8;
            const int64_t gm = m0 + r;
            ra[p] = gm < M ? *(const u32x4s*)(A + gm * K + k0 + kk) : u32x4s{0u, 0u, 0u, 0u};
            rb[p] = n0 + r < N ? *(const u32x4s*)(W + (int64_t)(n0 + r) * K + k0 + kk) : u32x4s{0u, 0u, 0u, 0u};
        }
    };
    fetch(0);
    for (int k0 = 0; k0 < K; k0 += kGK) {
        __syncthreads();                      // the previous step's operands are consumed
#pragma unroll
        for (int p = 0; p < kGLoads; p++) {
            const int idx = t + p * kBlock;
            const int r = idx >> 3, kk = (idx & 7) * 8;
            *(u32x4s*)&As[r][kk] = ra[p];
            *(u32x4s*)&Bs[r][kk] = rb[p];
        }
        __syncthreads();
        if (k0 + kGK < K) fetch(k0 + kGK);
#pragma unroll
        for (int ks = 0; ks < kGK; ks += 16) {
            const int kq = ks + (lane >> 5) * 8;
            bf16x8 a[2], b[2];
#pragma unroll
            for (int i = 0; i < 2; i++) a[i] = *(const bf16x8*)&As[wm + i * 32 + (lane & 31)][kq];
#pragma unroll
            for (int i = 0; i < 2; i++) b[i] = *(const bf16x8*)&Bs[wn + i * 32 + (lane & 31)][kq];
#pragma unroll
            for (int i = 0; i < 2; i++)
#pragma unroll
                for (int jj = 0; jj < 2; jj++)
                    acc[i][jj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[jj], a[i], acc[i][jj], 0, 0, 0);
        }
    }
    // Epilogue through LDS: the tile (bias added, ReLU, converted) is written
    // there in the MFMA's layout and leaves as whole rows of 16-byte pieces, so
    // every line of Z is written by one store instruction (stored straight from
    // the MFMA layout, the partial lines doubled Z's HBM write traffic).  A
    // float tile is larger than the operand tiles, so it leaves in two passes of
    // 64 rows: rows i = 0 of every wave's quarter, then rows i = 1.  N is a
    // multiple of 32 (checked on the host), so a piece or a group of four
    // columns that starts inside Z ends inside it.
    typedef typename std::conditional<OUT_F32, float, uint16_t>::type OutT;
    constexpr int PASSES = OUT_F32 ? 2 : 1;
    constexpr int RP = kGM / PASSES;                    // tile rows per pass
    constexpr int CE = 16 / (int)sizeof(OutT);          // elements per 16-byte piece
    constexpr int CP = kGN + CE;                        // padded LDS row (elements)
    static_assert(RP * CP * sizeof(OutT) <= sizeof(smem), "the output tile fits the operand tiles' LDS");
    OutT (*Cs)[CP] = reinterpret_cast<OutT (*)[CP]>(smem);
#pragma unroll
    for (int pass = 0; pass < PASSES; pass++) {
        __syncthreads();                                // LDS is free: operands consumed, previous pass written out
#pragma unroll
        for (int i = 0; i < 2; i++) {
            if (PASSES == 2 && i != pass) continue;
            const int lrow = PASSES == 1 ? wm + i * 32 + (lane & 31) : (wm >> 1) + (lane & 31);
#pragma unroll
            for (int jj = 0; jj < 2; jj++)
#pragma unroll
                for (int g = 0; g < 4; g++) {
                    const int c = wn + jj * 32 + g * 8 + (lane >> 5) * 4;
                    if (n0 + c >= N) continue;
                    float z[4];
#pragma unroll
                    for (int e = 0; e < 4; e++) {
                        z[e] = acc[i][jj][g * 4 + e] + bias[n0 + c + e];
                        if (RELU) z[e] = z[e] > 0.f ? z[e] : 0.f;
                    }
                    if (OUT_F32) *(f32x4*)&Cs[lrow][c] = f32x4{z[0], z[1], z[2], z[3]};
                    else *(u16x4*)&Cs[lrow][c] = u16x4{to_bf16(z[0]), to_bf16(z[1]), to_bf16(z[2]), to_bf16(z[3])};
                }
        }
        __syncthreads();
        constexpr int PPR = kGN / CE;                   // pieces per tile row
#pragma unroll
        for (int q = 0; q < RP * PPR / kBlock; q++) {
            const int idx = t + q * kBlock, lrow = idx / PPR, c = (idx % PPR) * CE;
            const int r = PASSES == 1 ? lrow : (lrow / 32) * 64 + pass * 32 + lrow % 32;
            const int64_t gm = m0 + r;
            if (gm < M && n0 + c < N) *(u32x4s*)((OutT*)Z + gm * N + n0 + c) = *(const u32x4s*)&Cs[lrow][c];
        }
    }
}

template <typename InT, int LPR>
static void launch_agg_k(const void* hin, const LayerOffsets& o, const int32_t* row_ptr, const int32_t* col, int H,
                         int64_t M, int din, uint16_t* A, hipStream_t st) {
    constexpr int64_t per_wg = (int64_t)kWavesPerBlock * (kWave / LPR);
    const int G = (int)std::max<int64_t>(1, std::min<int64_t>((M + per_wg - 1) / per_wg, 1 << 20));
    AGNES_LAUNCH((k_sage_agg<InT, LPR>), dim3(G), dim3(kBlock), 0, st, (const InT*)hin, o, row_ptr, col, H, M,
                       din, A);
}

// Lanes per row: the largest power of two up to 64 that the row's 16-byte
// pieces fill (din is a multiple of 32, so there are at least 4 pieces).
template <typename InT>
static void launch_agg(const void* hin, const LayerOffsets& o, const int32_t* row_ptr, const int32_t* col, int H,
                       int64_t M, int din, uint16_t* A, hipStream_t st) {
    const int pieces = din / In16<InT>::E;
    if (pieces >= 64) launch_agg_k<InT, 64>(hin, o, row_ptr, col, H, M, din, A, st);
    else if (pieces >= 32) launch_agg_k<InT, 32>(hin, o, row_ptr, col, H, M, din, A, st);
    else if (pieces >= 16) launch_agg_k<InT, 16>(hin, o, row_ptr, col, H, M, din, A, st);
    else if (pieces >= 8) launch_agg_k<InT, 8>(hin, o, row_ptr, col, H, M, din, A, st);
    else launch_agg_k<InT, 4>(hin, o, row_ptr, col, H, M, din, A, st);
}

static void check_forward(const Batch& b, const agnes_sage_model& m, const float* out) {
    const Store& s = *b.store;
    AGNES_REQUIRE(b.state == kGathering || b.state == kDone, AGNES_ERR_INVALID, "the batch holds no finished hyperbatch");
    AGNES_REQUIRE(m.L == b.L, AGNES_ERR_INVALID, "the model needs one layer per hop of the batch");
    AGNES_REQUIRE(out, AGNES_ERR_INVALID, "out must not be NULL");
    for (int i = 0; i <= m.L; i++)
        AGNES_REQUIRE(m.dims[i] >= 32 && m.dims[i] <= 4096 && m.dims[i] % 32 == 0, AGNES_ERR_INVALID,
                      "dims must be positive multiples of 32, at most 4096");
    const int esz = s.feat_dtype == AGNES_FLOAT32 ? 4 : 2;
    AGNES_REQUIRE((int64_t)m.dims[0] * esz == s.row_bytes, AGNES_ERR_INVALID, "dims[0] must be the feature dim");
    for (int i = 0; i < m.L; i++) {
        AGNES_REQUIRE(m.weight[i] && m.bias[i], AGNES_ERR_INVALID, "weights and biases must not be NULL");
        AGNES_REQUIRE(((uintptr_t)m.weight[i] & 15) == 0, AGNES_ERR_INVALID, "weights must be 16-byte aligned");
    }
    AGNES_REQUIRE(((uintptr_t)out & 15) == 0, AGNES_ERR_INVALID, "out must be 16-byte aligned");
}

// Destination rows of layer i (hop L-1-i) over the hyperbatch, and the largest
// [h ; mean] matrix and hidden output (elements) of the forward.
struct ForwardSizes {
    int64_t M[AGNES_MAX_LAYERS];
    int64_t Amax, Hmax;
};

static ForwardSizes forward_sizes(const Batch& b, const agnes_sage_model& m) {
    ForwardSizes z{};
    z.Hmax = 1;
    const int H = b.H, L = b.L;
    for (int i = 0; i < L; i++) {
        const int l = L - 1 - i;
        int64_t M = 0;
        for (int j = 0; j < H; j++) M += b.layer_sizes[(size_t)j * (L + 1) + l];
        z.M[i] = M;
        z.Amax = std::max(z.Amax, M * 2 * m.dims[i]);
        if (i + 1 < L) z.Hmax = std::max(z.Hmax, M * m.dims[i + 1]);
    }
    return z;
}

// The forward's kernels on st: per layer the aggregation into A, then the GEMM
// (into hidden[i & 1], or into out for the last layer).  doffs holds the
// layers' offsets, [L][4][H+1] int64 (d_off, in_off, rp_off, col_off).
static void enqueue_forward(const Batch& b, const agnes_sage_model& m, const ForwardSizes& z, const int64_t* doffs,
                            uint16_t* A, void* const hidden[2], float* out, hipStream_t st) {
    const Store& s = *b.store;
    const int H = b.H, L = b.L;
    const void* hin = b.features.ptr;
    for (int i = 0; i < L; i++) {
        const int l = L - 1 - i;
        LayerOffsets o{doffs + ((size_t)i * 4 + 0) * (H + 1), doffs + ((size_t)i * 4 + 1) * (H + 1),
                       doffs + ((size_t)i * 4 + 2) * (H + 1), doffs + ((size_t)i * 4 + 3) * (H + 1)};
        const int din = m.dims[i], dout = m.dims[i + 1];
        const int64_t M = z.M[i];
        if (M == 0) continue;
        if (i == 0 && s.feat_dtype == AGNES_FLOAT32)
            launch_agg<float>(hin, o, b.row_ptr[l].as<int32_t>(), b.col[l].as<int32_t>(), H, M, din, A, st);
        else if (i == 0 && s.feat_dtype == AGNES_FLOAT16)
            launch_agg<_Float16>(hin, o, b.row_ptr[l].as<int32_t>(), b.col[l].as<int32_t>(), H, M, din, A, st);
        else
            launch_agg<uint16_t>(hin, o, b.row_ptr[l].as<int32_t>(), b.col[l].as<int32_t>(), H, M, din, A, st);
        const int64_t mbs = (M + kGM - 1) / kGM, nbs = (dout + kGN - 1) / kGN;
        const dim3 grid((unsigned)((mbs + 7) / 8 * 8 * nbs));
        if (i + 1 < L) {
            void* zout = hidden[i & 1];
            AGNES_LAUNCH((k_sage_gemm<true, false>), grid, dim3(kBlock), 0, st, A,
                         (const uint16_t*)m.weight[i], m.bias[i], M, dout, 2 * din, zout);
            hin = zout;
        } else {
            AGNES_LAUNCH((k_sage_gemm<false, true>), grid, dim3(kBlock), 0, st, A,
                         (const uint16_t*)m.weight[i], m.bias[i], M, dout, 2 * din, (void*)out);
        }
    }
}

void sage_forward(Batch& b, const agnes_sage_model& m, float* out, hipStream_t st) {
    Range range("agnes_sage_forward");
    check_forward(b, m, out);
    const int H = b.H, L = b.L;
    const ForwardSizes z = forward_sizes(b, m);
    // host offsets of every layer: d_off, in_off, rp_off, col_off ([H+1] each)
    std::vector<int64_t> offs((size_t)L * 4 * (H + 1));
    for (int i = 0; i < L; i++) {
        const int l = L - 1 - i;
        int64_t* d_off = &offs[((size_t)i * 4 + 0) * (H + 1)];
        int64_t* in_off = &offs[((size_t)i * 4 + 1) * (H + 1)];
        int64_t* rp = &offs[((size_t)i * 4 + 2) * (H + 1)];
        int64_t* co = &offs[((size_t)i * 4 + 3) * (H + 1)];
        d_off[0] = 0;
        for (int j = 0; j < H; j++) d_off[j + 1] = d_off[j] + b.layer_sizes[(size_t)j * (L + 1) + l];
        for (int j = 0; j <= H; j++) {
            in_off[j] = i == 0 ? b.node_off[j] : offs[((size_t)(i - 1) * 4 + 0) * (H + 1) + j];
            rp[j] = b.rp_off[l][j];
            co[j] = b.col_off[l][j];
        }
    }
    if (b.sage_ev) AGNES_CHECK_HIP(hipEventSynchronize(b.sage_ev));   // the previous upload has left the pinned buffer
    else AGNES_CHECK_HIP(hipEventCreateWithFlags(&b.sage_ev, hipEventDisableTiming));
    if (!b.sage_done) AGNES_CHECK_HIP(hipEventCreateWithFlags(&b.sage_done, hipEventDisableTiming));
    // a previous forward on another stream still reads the scratch rows this
    // one overwrites
    if (b.sage_pending) AGNES_CHECK_HIP(hipStreamWaitEvent(st, b.sage_done, 0));
    b.sage_host.reserve(offs.size() * 8);
    memcpy(b.sage_host.ptr, offs.data(), offs.size() * 8);
    b.sage_off.reserve(offs.size() * 8);
    // sizes vary by hyperbatch: headroom keeps reallocations (and the device
    // synchronisation of the free that comes with each) rare
    b.sage_a.reserve_slack((size_t)std::max<int64_t>(z.Amax, 1) * 2);
    for (int k = 0; k < 2; k++) b.sage_h[k].reserve_slack((size_t)z.Hmax * 2);
    if (st != b.stream) AGNES_CHECK_HIP(hipStreamWaitEvent(st, b.gathered_at, 0));
    AGNES_CHECK_HIP(hipMemcpyAsync(b.sage_off.ptr, b.sage_host.ptr, offs.size() * 8, hipMemcpyHostToDevice, st));
    AGNES_CHECK_HIP(hipEventRecord(b.sage_ev, st));
    void* const hidden[2] = {b.sage_h[0].ptr, b.sage_h[1].ptr};
    enqueue_forward(b, m, z, b.sage_off.as<int64_t>(), b.sage_a.as<uint16_t>(), hidden, out, st);
    // what the next hyperbatch or forward on this batch waits for
    AGNES_CHECK_HIP(hipEventRecord(b.sage_done, st));
    b.sage_pending = true;
}

// ----------------------------------------------------------------- no allocation

// Scratch space of agnes_sage_forward_noalloc: one array per GPU, held by the
// loaded code object until the process ends.  Host code never uses this name
// as an address; it uses the device address that hipGetSymbolAddress returns
// for the current device (scratch_on_device).
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

static void* scratch_on_device(int dev) {
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static void* addr[kMaxDevices] = {};
    AGNES_REQUIRE(dev >= 0 && dev < kMaxDevices, AGNES_ERR_INVALID, "device index out of range");
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void* p = nullptr;
        AGNES_CHECK_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        AGNES_REQUIRE(p, AGNES_ERR_DEVICE, "no device address for the scratch array");
        addr[dev] = p;
    }
    return addr[dev];
}

// The layers' offsets ([L][4][H+1], as enqueue_forward reads them) from the
// batch's device-side layer sizes [H][L+1], edge counts [H][L] and output row
// offsets node_off [H+1]: one workgroup, per layer and array an exclusive
// scan over the minibatches.
__global__ __launch_bounds__(kBlock) void k_sage_offsets(const int32_t* lsz, const int64_t* ecount,
                                                         const int64_t* node_off, int H, int L, int64_t* offs) {
    __shared__ int64_t lds[kWavesPerBlock];
    for (int i = 0; i < L; i++) {
        const int l = L - 1 - i;
        int64_t* d_off = offs + ((size_t)i * 4 + 0) * (H + 1);
        int64_t* in_off = offs + ((size_t)i * 4 + 1) * (H + 1);
        int64_t* rp = offs + ((size_t)i * 4 + 2) * (H + 1);
        int64_t* co = offs + ((size_t)i * 4 + 3) * (H + 1);
        const int64_t* prev_d = i > 0 ? offs + ((size_t)(i - 1) * 4 + 0) * (H + 1) : node_off;
        int64_t cd = 0, cr = 0, cc = 0;
        for (int base = 0; base < H; base += kBlock) {
            const int j = base + threadIdx.x;
            const int64_t n = j < H ? (int64_t)lsz[(int64_t)j * (L + 1) + l] : 0;
            const int64_t e = j < H ? ecount[(int64_t)j * L + l] : 0;
            int64_t t;
            const int64_t xd = block_exclusive_scan(n, lds, t);
            if (j < H) d_off[j] = cd + xd;
            cd += t;
            const int64_t xr = block_exclusive_scan(j < H ? n + 1 : (int64_t)0, lds, t);
            if (j < H) rp[j] = cr + xr;
            cr += t;
            const int64_t xc = block_exclusive_scan(e, lds, t);
            if (j < H) co[j] = cc + xc;
            cc += t;
        }
        if (threadIdx.x == 0) {
            d_off[H] = cd;
            rp[H] = cr;
            co[H] = cc;
        }
        __syncthreads();
        for (int j = threadIdx.x; j <= H; j += kBlock) in_off[j] = prev_d[j];
        __syncthreads();
    }
}

static size_t align256(size_t x) { return (x + 255) / 256 * 256; }

void sage_forward_noalloc(Batch& b, const agnes_sage_model& m, float* out, hipStream_t st) {
    Range range("agnes_sage_forward_noalloc");
    check_forward(b, m, out);
    const int H = b.H, L = b.L;
    const ForwardSizes z = forward_sizes(b, m);
    const size_t off_bytes = align256((size_t)L * 4 * (H + 1) * sizeof(int64_t));
    const size_t a_bytes = align256((size_t)std::max<int64_t>(z.Amax, 1) * 2);
    const size_t h_bytes = align256((size_t)z.Hmax * 2);
    const size_t need = off_bytes + a_bytes + 2 * h_bytes;
    AGNES_REQUIRE(need <= kNoAllocScratchBytes, AGNES_ERR_RANGE,
                  "the forward needs " + std::to_string(need) + " bytes of scratch; the no-allocation forward has " +
                      std::to_string(kNoAllocScratchBytes));
    int dev = 0;
    AGNES_CHECK_HIP(hipGetDevice(&dev));
    AGNES_REQUIRE(dev == b.store->device, AGNES_ERR_INVALID, "the current device is not the batch's device");
    char* base = (char*)scratch_on_device(dev);
    int64_t* offs = (int64_t*)base;
    uint16_t* A = (uint16_t*)(base + off_bytes);
    void* const hidden[2] = {base + off_bytes + a_bytes, base + off_bytes + a_bytes + h_bytes};
    if (st != b.stream) AGNES_CHECK_HIP(hipStreamWaitEvent(st, b.gathered_at, 0));
    AGNES_LAUNCH(k_sage_offsets, dim3(1), dim3(kBlock), 0, st, b.d_lsz, b.d_ecount, b.ws.mb_off.as<int64_t>(), H,
                 L, offs);
    enqueue_forward(b, m, z, offs, A, hidden, out, st);
    // what the next hyperbatch on this batch waits for (created with the batch)
    AGNES_CHECK_HIP(hipEventRecord(b.sage_done, st));
    b.sage_pending = true;
}

}  // namespace agnes
