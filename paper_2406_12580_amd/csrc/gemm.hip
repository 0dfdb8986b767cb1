// Matrix-core products of the library (gfx950).
//
// Gate projections of the BD-LRU (RecBLR, arXiv 2406.12580, section 3.2):
//   z_r = x W_r^T + b_r,  z_i = x W_i^T + b_i            (forward)
//   dx += dz_r W_r + dz_i W_i                            (backward, data)
//   dW_r = dz_r^T x, dW_i = dz_i^T x, db = sum_rows dz   (backward, weights)
// with the two gates handled as one concatenated operand of width 2D.  x and
// the weights use the I/O type; z and dz are fp32 scratch (rounding them to
// bf16 would cost about 1e-2 of relative accuracy in dW).
//
// Two engines:
//  * fastmm (namespace below, staging in mfma_tile.hpp), taken for every
//    shape with D % 8 == 0 and 16-byte-aligned operands: a 256-thread
//    workgroup owns a 128 x 128 output tile, each wave a 64 x 64 quarter as
//    4 x 4 blocks of v_mfma_f32_16x16x32_bf16 with fp32 accumulation.  K-slices
//    of 64 are fetched through buffer resources as 16-byte quads one slice
//    ahead (pinned with a scheduling barrier), fp32 operands split into bf16
//    hi and lo planes (a product becomes hi*hi + hi*lo + lo*hi), and stored to
//    LDS K-contiguous with a chunk swizzle that keeps fragment reads
//    conflict-free.  Tiles are numbered so that each XCD owns a contiguous run
//    of row blocks (their column tiles share that XCD's L2).  The weight
//    gradient is split over rows into about two workgroups per CU, its fp32
//    partials summed afterwards in a fixed order (deterministic), db summed
//    from the same staged dz rows.  The same engine packs the weights for the
//    fused scans (pack_group_kernel) and runs the decode step's product
//    (step_kernel), and its fp32 linear32 / wgrad kernels serve the model
//    step's linear layers.
//  * the generic kernels (proj_*_kernel), for D % 8 != 0 or unaligned
//    operands: 64 x 64 tiles, each wave a 32 x 32 quarter as 2 x 2 blocks of
//    v_mfma_f32_16x16x4_f32 (or 16x16x32_bf16 when both operands are bf16
//    inputs), one element per load, split-K weight gradient with a
//    fixed-order sum.
#include <initializer_list>
#include <type_traits>

#include "device_common.hpp"
#include "gemm.hpp"
#include "mfma_tile.hpp"

namespace recblr {

namespace {
constexpr int kTM = 64, kTN = 64, kThreads = 256;
}

typedef float f4v __attribute__((ext_vector_type(4)));
typedef __bf16 bf8v __attribute__((ext_vector_type(8)));

// ------------------------------------------------------------------ operand accessors
// a(i, k) and b(k, n) read one element; kAKFast / kBKFast say whether k is the
// contiguous index of the operand in memory (then k runs fastest across
// threads when staging, else i / n does).
// Forward: A = x [M x D], B(k, n) = Wcat[n][k] with Wcat = [W_r; W_i] ([2D x D]).
template <typename T>
struct FwdOps {
    static constexpr bool kAKFast = true, kBKFast = true;
    const T* x;
    const T* wr;
    const T* wi;
    int64_t D;
    __device__ float a(int64_t i, int64_t k) const { return load(x + i * D + k); }
    __device__ float b(int64_t k, int64_t n) const {
        return n < D ? load(wr + n * D + k) : load(wi + (n - D) * D + k);
    }
};

// Backward data: A(i, k) = [dz_r | dz_i][i][k] ([M x 2D]), B(k, n) = Wcat[k][n].
template <typename T>
struct DxOps {
    static constexpr bool kAKFast = true, kBKFast = false;
    const float* dzr;
    const float* dzi;
    const T* wr;
    const T* wi;
    int64_t D;
    __device__ float a(int64_t i, int64_t k) const {
        return k < D ? dzr[i * D + k] : dzi[i * D + (k - D)];
    }
    __device__ float b(int64_t k, int64_t n) const {
        return k < D ? load(wr + k * D + n) : load(wi + (k - D) * D + n);
    }
};

// Backward weights: A(o, row) = [dz_r | dz_i][row][o] ([2D x M]),
// B(row, k) = x[row][k] for k < D and 1 for k = D (so column D yields db).
template <typename T>
struct DwOps {
    static constexpr bool kAKFast = false, kBKFast = false;
    const float* dzr;
    const float* dzi;
    const T* x;
    int64_t D;
    __device__ float a(int64_t o, int64_t row) const {
        return o < D ? dzr[row * D + o] : dzi[row * D + (o - D)];
    }
    __device__ float b(int64_t row, int64_t k) const {
        return k < D ? load(x + row * D + k) : 1.0f;
    }
};

// C tile = sum over k in [k_begin, k_end) of A(i, k) B(k, n) for the 64 x 64
// tile at (blockIdx.x * 64, blockIdx.y * 64); each result goes to
// epi(i, n, value).  BF16: both operands are bf16 values (exact in bf16) and
// the bf16 MFMA is used; otherwise fp32 MFMA.
template <bool BF16, class Ops, class Epi>
__device__ __forceinline__ void mfma_tile(const Ops& ops, int64_t M, int64_t N, int64_t k_begin,
                                          int64_t k_end, Epi epi) {
    using E = typename std::conditional<BF16, __bf16, float>::type;
    constexpr int kBK = BF16 ? 32 : 16;       // K-slice staged per iteration
    constexpr int kPad = BF16 ? 8 : 1;        // keeps 16-byte rows (bf16) / spreads banks (fp32)
    __shared__ __attribute__((aligned(16))) E As[kTM][kBK + kPad];
    __shared__ __attribute__((aligned(16))) E Bs[kTN][kBK + kPad];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wv = tid >> 6;
    const int wm = wv >> 1, wn = wv & 1;      // this wave's 32 x 32 quarter
    const int64_t i0 = (int64_t)blockIdx.x * kTM, n0 = (int64_t)blockIdx.y * kTN;
    f4v acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f4v{0.0f, 0.0f, 0.0f, 0.0f};

    for (int64_t k0 = k_begin; k0 < k_end; k0 += kBK) {
        for (int e = tid; e < kTM * kBK; e += kThreads) {
            const int ii = Ops::kAKFast ? e / kBK : e % kTM;
            const int kk = Ops::kAKFast ? e % kBK : e / kTM;
            const int64_t i = i0 + ii, k = k0 + kk;
            As[ii][kk] = (E)((i < M && k < k_end) ? ops.a(i, k) : 0.0f);
        }
        for (int e = tid; e < kTN * kBK; e += kThreads) {
            const int nn = Ops::kBKFast ? e / kBK : e % kTN;
            const int kk = Ops::kBKFast ? e % kBK : e / kTN;
            const int64_t n = n0 + nn, k = k0 + kk;
            Bs[nn][kk] = (E)((n < N && k < k_end) ? ops.b(k, n) : 0.0f);
        }
        __syncthreads();
        if constexpr (BF16) {
            // v_mfma_f32_16x16x32_bf16: lane l supplies row l%16, k = 8*(l/16)..+7.
            bf8v av[2], bv[2];
#pragma unroll
            for (int i = 0; i < 2; ++i)
                av[i] = *(const bf8v*)&As[wm * 32 + i * 16 + (lane & 15)][8 * (lane >> 4)];
#pragma unroll
            for (int j = 0; j < 2; ++j)
                bv[j] = *(const bf8v*)&Bs[wn * 32 + j * 16 + (lane & 15)][8 * (lane >> 4)];
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[i], bv[j], acc[i][j],
                                                                         0, 0, 0);
        } else {
            // v_mfma_f32_16x16x4_f32: lane l supplies row l%16, k = l/16.
#pragma unroll
            for (int ks = 0; ks < kBK; ks += 4) {
                float av[2], bv[2];
#pragma unroll
                for (int i = 0; i < 2; ++i)
                    av[i] = As[wm * 32 + i * 16 + (lane & 15)][ks + (lane >> 4)];
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    bv[j] = Bs[wn * 32 + j * 16 + (lane & 15)][ks + (lane >> 4)];
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i], bv[j],
                                                                          acc[i][j], 0, 0, 0);
            }
        }
        __syncthreads();
    }
    // D[r][c] of a 16 x 16 block: lane l holds rows 4*(l/16)+v, column l%16.
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int64_t r = i0 + wm * 32 + i * 16 + 4 * (lane >> 4) + v;
                const int64_t c = n0 + wn * 32 + j * 16 + (lane & 15);
                if (r < M && c < N) epi(r, c, acc[i][j][v]);
            }
}

template <typename T>
__global__ __launch_bounds__(kThreads) void proj_fwd_kernel(const T* x, const T* wr,
                                                            const T* br, const T* wi,
                                                            const T* bi, float* zr, float* zi,
                                                            int64_t M, int64_t D) {
    FwdOps<T> ops{x, wr, wi, D};
    mfma_tile<sizeof(T) == 2>(ops, M, 2 * D, 0, D, [&](int64_t i, int64_t n, float v) {
        if (n < D) {
            store(zr + i * D + n, v + (br ? load(br + n) : 0.0f));
        } else {
            int64_t o = n - D;
            store(zi + i * D + o, v + (bi ? load(bi + o) : 0.0f));
        }
    });
}

template <typename T, typename TD = T>
__global__ __launch_bounds__(kThreads) void proj_dx_kernel(const float* dzr, const float* dzi,
                                                           const T* wr, const T* wi, TD* dx,
                                                           int64_t M, int64_t D) {
    DxOps<T> ops{dzr, dzi, wr, wi, D};
    mfma_tile<false>(ops, M, D, 0, 2 * D, [&](int64_t i, int64_t n, float v) {
        TD* p = dx + i * D + n;
        store(p, load(p) + v);  // dx already holds the direct term delta * beta
    });
}

// Split-K partial of [dW_r; dW_i | db]: partial[split][o][k], o < 2D, k <= D.
template <typename T>
__global__ __launch_bounds__(kThreads) void proj_dw_kernel(const float* dzr, const float* dzi,
                                                           const T* x, float* partial,
                                                           int64_t M, int64_t D,
                                                           int64_t rows_per_split) {
    DwOps<T> ops{dzr, dzi, x, D};
    const int64_t split = blockIdx.z;
    const int64_t k_begin = split * rows_per_split;
    int64_t k_end = k_begin + rows_per_split;
    if (k_end > M) k_end = M;
    const int64_t N = D + 1;
    float* out = partial + split * (2 * D) * N;
    mfma_tile<false>(ops, 2 * D, N, k_begin, k_end,
                     [&](int64_t o, int64_t k, float v) { out[o * N + k] = v; });
}

// Sum the split-K partials in split order (fp64) into dW_r, dW_i, db_r, db_i.
__global__ void proj_dw_reduce_kernel(const float* partial, int64_t splits, int64_t D,
                                      float* dwr, float* dbr, float* dwi, float* dbi) {
    const int64_t N = D + 1;
    const int64_t total = 2 * D * N;
    int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= total) return;
    double s = 0.0;
    for (int64_t k = 0; k < splits; ++k) s += (double)partial[k * total + e];
    int64_t o = e / N, c = e % N;
    float v = (float)s;
    if (o < D) {
        if (c < D) dwr[o * D + c] = v;
        else dbr[o] = v;
    } else {
        if (c < D) dwi[(o - D) * D + c] = v;
        else dbi[o - D] = v;
    }
}

// ------------------------------------------------------------------ fast path
// Taken when D % 8 == 0, the operands are 16-byte aligned and every operand
// spans less than 2 GiB (all workload shapes of the paper).  A 256-thread
// workgroup computes a 128 x 128 tile of C = A B^T (A: rows m, B: rows n, both
// over the contracted index k); each wave owns a 64 x 64 quarter as 4 x 4
// blocks of v_mfma_f32_16x16x32_bf16.  An fp32 operand is split into
// hi = bf16(v) and lo = bf16(v - hi) and a product of two fp32 operands is
// formed from the three terms hi*hi + hi*lo + lo*hi (a bf16 operand is exact
// and needs one plane): each product then carries a relative error below
// 3 * 2^-17 against 2^-24 for a plain fp32 product, while the matrix cores
// deliver 16x the fp32 MFMA rate, so the projection stays bound by HBM
// instead of by fp32 MFMA.  The weights are packed once per call into bf16
// planes laid out the way the tiles read them.
//
// Operands are read through buffer resources at per-lane 32-bit byte
// offsets computed once per tile; offsets at or past a resource's size read
// zero, which masks the contraction tail.  Operand quads (4 consecutive
// elements along the contiguous memory index) for the next K-slice are
// loaded into registers while the current slice is multiplied from LDS.
// Tiles are numbered so that consecutive tiles of one row block land on the
// same XCD and share its L2.
namespace fastmm {

// Multiplies the staged 128 x BK slices: the wave's 4 x 4 blocks of 16 x 16,
// k-steps of 32.  Lane l supplies row l % 16 and k = 8 (l / 16) .. +7 of
// each fragment (the k order inside a step is irrelevant to the sum as long
// as A and B use the same one).
template <int PA, int PB>
__device__ __forceinline__ void mma_slice(__bf16 (*la)[BM][KP], __bf16 (*lb)[BN][KP],
                                          f4 (&acc)[4][4], int wm, int wn, int fr, int fk) {
#pragma unroll
    for (int ks = 0; ks < BK; ks += 32) {
        b8 fa[PA][4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int ra = wm * 64 + i * 16 + fr;
#pragma unroll
            for (int p = 0; p < PA; ++p) fa[p][i] = *(const b8*)&la[p][ra][lds_col(ra, ks + fk)];
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int rb = wn * 64 + j * 16 + fr;
            b8 fb[PB];
#pragma unroll
            for (int p = 0; p < PB; ++p) fb[p] = *(const b8*)&lb[p][rb][lds_col(rb, ks + fk)];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                if constexpr (PB == 2)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[0][i], fb[1],
                                                                         acc[i][j], 0, 0, 0);
                if constexpr (PA == 2)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[1][i], fb[0],
                                                                         acc[i][j], 0, 0, 0);
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[0][i], fb[0], acc[i][j],
                                                                     0, 0, 0);
            }
        }
    }
}

// Epilogue staging: each wave passes its 64 x 64 result through LDS in strips
// of 16 rows (pitch 68 floats: conflict-free writes in the MFMA layout) and
// then hands each lane four float4 of one row segment, so global accesses are
// 256-byte row segments.
constexpr int EP = 68;
constexpr size_t kEpiBytes = 4 * 16 * EP * sizeof(float);
template <int PA, int PB>
constexpr size_t lds_bytes() {
    const size_t tiles = (size_t)(PA * BM + PB * BN) * KP * 2;
    return tiles > kEpiBytes ? tiles : kEpiBytes;
}

// Rows of strip i handled by this lane in the epilogue: four rows 4 apart.
__device__ __forceinline__ void strip_rows(int64_t m0w, int i, int lane, int64_t (&m)[4]) {
#pragma unroll
    for (int q = 0; q < 4; ++q) m[q] = m0w + i * 16 + 4 * q + (lane >> 4);
}

// Epilogues without a read of the destination.
struct NoPre {};

// Passes the wave's 64 x 64 accumulator block (rows m0w.., columns n0w..)
// to epi.run(m[4], n, v[4], pre): four row indices, the first of four columns,
// the four float4 values, and what epi.load fetched.  With kStripLoads,
// epi.load fetches per strip (strip 0's comes in as `pre`, strip i + 1's is
// fetched before strip i is stored); otherwise `pre` serves every strip.
// Every thread of the workgroup must call it.
template <class Epi>
__device__ __forceinline__ void tile_epilogue(const f4 (&acc)[4][4], char* smem, int64_t m0w,
                                              int64_t n0w, const Epi& epi,
                                              typename Epi::pre_t pre) {
    const int lane = threadIdx.x & 63;
    float* buf = (float*)smem + (threadIdx.x >> 6) * 16 * EP;
    const int64_t n = n0w + 4 * (lane & 15);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        // MFMA result layout: lane l holds rows 4 (l / 16) + v, column l % 16 of a block.
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                buf[(4 * (lane >> 4) + v) * EP + j * 16 + (lane & 15)] = acc[i][j][v];
        __syncthreads();
        int64_t m[4];
        strip_rows(m0w, i, lane, m);
        f4 val[4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
            val[q] = *(const f4*)&buf[(4 * q + (lane >> 4)) * EP + 4 * (lane & 15)];
        if constexpr (Epi::kStripLoads) {
            // The next strip's reads go out before this strip's stores: vector
            // memory operations complete in issue order, so a read issued
            // after a store could only be waited for together with the store.
            typename Epi::pre_t next{};
            if (i < 3) {
                int64_t mn[4];
                strip_rows(m0w, i + 1, lane, mn);
                epi.load(mn, n, next);
            }
            epi.run(m, n, val, pre);
            pre = next;
        } else {
            epi.run(m, n, val, pre);
        }
        __syncthreads();
    }
}

// One output tile at (m0, n0): the sum over k in [k_begin, k_end) of
// A(m, k) B(n, k), handed to epi.  The next K-slice is loaded during the
// current slice's MFMAs, and during the last slice the epilogue's reads of
// the destination.  If colsum_out is not null (A not KFAST), the sums over the
// same k range of the tile's 128 rows of A are written there.
template <class OpA, class OpB, class Epi>
__device__ __forceinline__ void tile(const OpA& a, const OpB& b, int64_t m0, int64_t n0,
                                     int64_t k_begin, int64_t k_end, const Epi& epi, char* smem,
                                     float* colsum_out = nullptr) {
    constexpr int PA = OpA::kPlanes, PB = OpB::kPlanes;
    __bf16 (*la)[BM][KP] = (__bf16 (*)[BM][KP])smem;
    __bf16 (*lb)[BN][KP] = (__bf16 (*)[BN][KP])(smem + (size_t)PA * BM * KP * 2);
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wv = tid >> 6;
    const int wm = wv >> 1, wn = wv & 1;
    const int fr = lane & 15, fk = 8 * (lane >> 4);
    const int64_t m0w = m0 + wm * 64, n0w = n0 + wn * 64;
    const int64_t nsl = k_end > k_begin ? (k_end - k_begin + BK - 1) / BK : 0;

    const Stager<OpA> sa(a, m0, tid);
    const Stager<OpB> sb(b, n0, tid);
    typename OpA::raw_t ra[NQ];
    typename OpB::raw_t rb[NQ];
    f4 cs = f4{0.0f, 0.0f, 0.0f, 0.0f};
    f4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    typename Epi::pre_t pre{};
    int64_t mr[4];
    strip_rows(m0w, 0, lane, mr);
    const int64_t ne = n0w + 4 * (lane & 15);

    if (nsl == 0) {
        epi.load(mr, ne, pre);
    } else {
        sa.fetch(a, k_begin, k_end, tid, ra);
        sb.fetch(b, k_begin, k_end, tid, rb);
        for (int64_t sl = 0; sl + 1 < nsl; ++sl) {
            store_slice<OpA>(la, tid, ra);
            store_slice<OpB>(lb, tid, rb);
            if constexpr (!OpA::kKFast)
                if (colsum_out) add_colsum(cs, ra);
            __syncthreads();
            const int64_t k0 = k_begin + (sl + 1) * BK;
            sa.fetch(a, k0, k_end, tid, ra);
            sb.fetch(b, k0, k_end, tid, rb);
            // Keep the loads ahead of the MFMAs: left to itself the scheduler
            // sinks them below the multiplications (reusing fragment
            // registers), and the next slice then waits for a full memory
            // round trip.
            __builtin_amdgcn_sched_barrier(0);
            mma_slice<PA, PB>(la, lb, acc, wm, wn, fr, fk);
            __syncthreads();
        }
        store_slice<OpA>(la, tid, ra);
        store_slice<OpB>(lb, tid, rb);
        if constexpr (!OpA::kKFast)
            if (colsum_out) add_colsum(cs, ra);
        __syncthreads();
        epi.load(mr, ne, pre);
        __builtin_amdgcn_sched_barrier(0);
        mma_slice<PA, PB>(la, lb, acc, wm, wn, fr, fk);
        __syncthreads();
    }
    if (!OpA::kKFast && colsum_out) {
        // Reduce the 8 k-groups of each column quad through LDS.
        f4* red = (f4*)smem;
        red[tid] = cs;
        __syncthreads();
        if (tid < 32) {
            f4 v = red[tid];
#pragma unroll
            for (int g = 1; g < 8; ++g) v += red[tid + 32 * g];
#pragma unroll
            for (int q = 0; q < 4; ++q) colsum_out[4 * tid + q] = v[q];
        }
        __syncthreads();
    }
    if constexpr (Epi::kOwnStore)
        epi.store_tile(acc, m0w, n0w, pre);
    else
        tile_epilogue(acc, smem, m0w, n0w, epi, pre);
}

// Logical tile of this workgroup: the hardware deals consecutive workgroup ids
// round-robin over the 8 XCDs; this renumbering gives each XCD a contiguous
// run of logical tiles.  Returns -1 for the padding workgroups.
__device__ __forceinline__ int64_t xcd_tile(int64_t tiles) {
    const int64_t padded = (tiles + 7) & ~(int64_t)7;
    const int64_t w = blockIdx.x;
    const int64_t t = (w & 7) * (padded >> 3) + (w >> 3);
    return t < tiles ? t : -1;
}

inline unsigned grid_of(int64_t tiles) { return (unsigned)((tiles + 7) & ~(int64_t)7); }

// ---- weight packing: bf16 planes (hi, and lo = bf16(w - hi) for fp32 weights)
// of Wcat = [W_r; W_i] ([2D x D]) in the layouts the tiles read:
//   forward: P[n][k] = Wcat[n][k] (n < 2D, k < D)
//   dx:      P[n][k] = Wcat[k][n] (n < D, k < 2D)
template <typename T, bool TRANSPOSED>
__global__ __launch_bounds__(256) void pack_kernel(const T* wr, const T* wi, __bf16* out,
                                                   int64_t D) {
    const int64_t total = 2 * D * D;
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= total) return;
    int64_t row, col;  // element of Wcat
    if (TRANSPOSED) {
        const int64_t n = e / (2 * D), k = e % (2 * D);
        row = k;
        col = n;
    } else {
        row = e / D;
        col = e % D;
    }
    const float v = row < D ? to_f32(wr[row * D + col]) : to_f32(wi[(row - D) * D + col]);
    const __bf16 hi = (__bf16)v;
    out[e] = hi;
    if (sizeof(T) == 4) out[total + e] = (__bf16)(v - (float)hi);
}

// Weights ordered by channel group for the scan forward with the projections
// fused in: rows 128 g .. 128 g + 63 are W_r rows of channels 64 g .. 64 g + 63,
// the next 64 rows the W_i rows of the same channels (D % 64 == 0).
template <typename T>
__global__ __launch_bounds__(256) void pack_group_kernel(const T* wr, const T* wi, __bf16* out,
                                                         int64_t D) {
    const int64_t total = 2 * D * D;
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= total) return;
    const int64_t n = e / D, k = e % D;
    const int64_t ch = (n / 128) * 64 + n % 64;
    const float v = (n / 64) % 2 == 0 ? to_f32(wr[ch * D + k]) : to_f32(wi[ch * D + k]);
    const __bf16 hi = (__bf16)v;
    out[e] = hi;
    if (sizeof(T) == 4) out[total + e] = (__bf16)(v - (float)hi);
}

template <typename T>
struct FwdEpi {
    static constexpr bool kOwnStore = false;
    static constexpr bool kStripLoads = false;
    struct pre_t {
        float br[4], bi[4];  // the lane's four columns in both biases (one of them is 0)
    };
    float* zr;
    float* zi;
    const T* br;
    const T* bi;
    int64_t M, D;
    __device__ void load(const int64_t (&)[4], int64_t n, pre_t& pre) const {
        const ElemReader<T> rr(br, D), ri(bi, D);
        const bool g = n < D;  // the four columns are in one gate (D % 4 == 0)
        const int64_t o = g ? n : n - D;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            pre.br[c] = rr(g ? o + c : -1);
            pre.bi[c] = ri(g ? -1 : o + c);
        }
    }
    __device__ void run(const int64_t (&m)[4], int64_t n, const f4 (&v)[4],
                        const pre_t& pre) const {
        if (n >= 2 * D) return;
        float* base = n < D ? zr + n : zi + (n - D);
        f4 bias;
#pragma unroll
        for (int c = 0; c < 4; ++c) bias[c] = pre.br[c] + pre.bi[c];
#pragma unroll
        for (int q = 0; q < 4; ++q)
            if (m[q] < M) *(f4*)(base + m[q] * D) = v[q] + bias;
    }
};

// One 128 x 128 tile of [z_r | z_i] (M x 2D) per workgroup; pack holds the
// forward weight planes.
template <typename T>
__global__ __launch_bounds__(256, 2) void fwd_kernel(const T* x, const __bf16* pack,
                                                     const T* br, const T* bi, float* zr,
                                                     float* zi, int64_t M, int64_t D) {
    constexpr bool F32 = sizeof(T) == 4;
    using OpA = Operand<F32 ? kF32 : kBf16, true>;
    using OpB = Operand<F32 ? kPack2 : kPack1, true>;
    __shared__ __attribute__((aligned(16))) char smem[lds_bytes<OpA::kPlanes, OpB::kPlanes>()];
    const int64_t ntn = (2 * D + BN - 1) / BN;
    const int64_t t = xcd_tile(((M + BM - 1) / BM) * ntn);
    if (t < 0) return;
    const uint32_t plane = (uint32_t)(2 * D * D * 2);
    const OpA a{resource(x, (uint32_t)(M * D * sizeof(T))), (uint32_t)(D * sizeof(T)), 0, 0, 0};
    const OpB b{resource(pack, OpB::kPlanes * plane), (uint32_t)(D * 2), 0, 0, plane};
    const FwdEpi<T> epi{zr, zi, br, bi, M, D};
    tile(a, b, (t / ntn) * BM, (t % ntn) * BN, 0, D, epi, smem);
}

template <typename T>
struct DxEpi {
    static constexpr bool kOwnStore = false;
    static constexpr bool kStripLoads = true;
    struct pre_t {
        f4 v[4];
    };
    T* dx;
    int64_t M, D;
    // Reads dx, which holds the direct term delta * beta on entry, through a
    // buffer resource (rows past M and columns past D read zero): no branch
    // around the loads.
    __device__ void load(const int64_t (&m)[4], int64_t n, pre_t& pre) const {
        const __amdgpu_buffer_rsrc_t r = resource(dx, (uint32_t)(M * D * sizeof(T)));
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const uint32_t off =
                (n < D && m[q] < M) ? (uint32_t)((m[q] * D + n) * sizeof(T)) : kOOB;
            if constexpr (sizeof(T) == 4) {
                const u4v w = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
                pre.v[q] = f4{__uint_as_float(w.x), __uint_as_float(w.y), __uint_as_float(w.z),
                              __uint_as_float(w.w)};
            } else {
                pre.v[q] = widen(__builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0));
            }
        }
    }
    __device__ void run(const int64_t (&m)[4], int64_t n, const f4 (&v)[4],
                        const pre_t& pre) const {
        if (n >= D) return;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if (m[q] >= M) continue;
            const f4 r = pre.v[q] + v[q];
            if constexpr (sizeof(T) == 4) {
                *(f4*)(dx + m[q] * D + n) = r;
            } else {
                uint2 w;
                w.x = bf16_pair(r[0], r[1]);
                w.y = bf16_pair(r[2], r[3]);
                *(uint2*)(dx + m[q] * D + n) = w;
            }
        }
    }
};

// One 128 x 128 tile of dx per workgroup: dx += [dz_r | dz_i] Wcat, with the
// two dz halves at dzr and dzr + hoff bytes and pack holding Wcat^T planes.
template <typename T, typename TD = T>
__global__ __launch_bounds__(256, 2) void dx_kernel(const float* dzr, uint32_t hoff,
                                                    const __bf16* pack, TD* dx, int64_t M,
                                                    int64_t D) {
    constexpr bool F32 = sizeof(T) == 4;  // fp32 weights: two bf16 planes
    using OpA = Operand<kF32, true, true>;
    using OpB = Operand<F32 ? kPack2 : kPack1, true>;
    __shared__ __attribute__((aligned(16))) char smem[lds_bytes<OpA::kPlanes, OpB::kPlanes>()];
    const int64_t ntn = (D + BN - 1) / BN;
    const int64_t t = xcd_tile(((M + BM - 1) / BM) * ntn);
    if (t < 0) return;
    const uint32_t plane = (uint32_t)(2 * D * D * 2);
    const OpA a{resource(dzr, hoff + (uint32_t)(M * D * 4)), (uint32_t)(D * 4), (uint32_t)D, hoff,
                0};
    const OpB b{resource(pack, OpB::kPlanes * plane), (uint32_t)(2 * D * 2), 0, 0, plane};
    const DxEpi<TD> epi{dx, M, D};
    tile(a, b, (t / ntn) * BM, (t % ntn) * BN, 0, 2 * D, epi, smem);
}

struct DwEpi {
    static constexpr bool kOwnStore = false;
    static constexpr bool kStripLoads = false;
    using pre_t = NoPre;
    float* out;
    int64_t O, D;
    __device__ void load(const int64_t (&)[4], int64_t, NoPre&) const {}
    __device__ void run(const int64_t (&m)[4], int64_t n, const f4 (&v)[4], NoPre) const {
        if (n >= D) return;
#pragma unroll
        for (int q = 0; q < 4; ++q)
            if (m[q] < O) *(f4*)(out + m[q] * D + n) = v[q];
    }
};

// Split-K partial of [dW_r; dW_i]: partial[split][o][k] (o < 2D, k < D), and
// of [db_r; db_i]: dbpart[split][o].  The dz halves are at dzr and dzr + hoff
// bytes.
template <typename T>
__global__ __launch_bounds__(256, 2) void dw_kernel(const float* dzr, uint32_t hoff, const T* x,
                                                    float* partial, float* dbpart, int64_t M,
                                                    int64_t D, int64_t splits,
                                                    int64_t rows_per_split) {
    // A(o, row) = dz[row][o], B(k, row) = x[row][k]: memory rows are the
    // contracted index for both.
    using OpA = Operand<kF32, false, true>;
    using OpB = Operand<sizeof(T) == 4 ? kF32 : kBf16, false>;
    __shared__ __attribute__((aligned(16))) char smem[lds_bytes<OpA::kPlanes, OpB::kPlanes>()];
    __shared__ float colsum[BM];
    const int64_t nto = (2 * D + BM - 1) / BM, ntn = (D + BN - 1) / BN;
    const int64_t t = xcd_tile(nto * ntn * splits);
    if (t < 0) return;
    const int64_t split = t / (nto * ntn), tl = t % (nto * ntn);
    const int64_t to = tl / ntn, tn = tl % ntn;
    const int64_t k_begin = split * rows_per_split;
    const int64_t k_end = k_begin + rows_per_split < M ? k_begin + rows_per_split : M;
    const OpA a{resource(dzr, hoff + (uint32_t)(M * D * 4)), (uint32_t)(D * 4), (uint32_t)D, hoff,
                0};
    const OpB b{resource(x, (uint32_t)(M * D * sizeof(T))), (uint32_t)(D * sizeof(T)), 0, 0, 0};
    const DwEpi epi{partial + split * (2 * D) * D, 2 * D, D};
    // The tiles of column block 0 also reduce db from the dz rows they stage.
    tile(a, b, to * BM, tn * BN, k_begin, k_end, epi, smem, tn == 0 ? colsum : nullptr);
    if (tn == 0) {
        const int64_t o = to * BM + threadIdx.x;
        if (threadIdx.x < BM && o < 2 * D) dbpart[split * 2 * D + o] = colsum[threadIdx.x];
    }
}

// ---- fp32 tiles (v_mfma_f32_16x16x4_f32), for products whose rounding must
// stay that of fp32: the forward products and data gradients of the model's
// linear layers (the 3-term bf16 split above moved the model's gradients by
// up to 3e-4 there).  Same 128 x 128 output tiles, 4-wave layout, epilogues
// and slice prefetch as above; both operands have the contracted index
// contiguous in memory (KFAST) and sit in LDS as fp32 rows of BK floats
// padded to KP32 (16-byte aligned rows; a fragment read of 8 consecutive
// rows touches 8 distinct bank groups).  Within a slice, lane group
// g = lane / 16 contracts k = 16 g .. 16 g + 15: MFMA step s takes
// k = 16 g + s for the four "k" inputs of the instruction, so that each lane
// reads its fragments as 16-byte vectors.
constexpr int KP32 = BK + 4;
constexpr size_t kLds32 = (size_t)(BM + BN) * KP32 * sizeof(float);

__device__ __forceinline__ void store_slice32(float (*lds)[KP32], int tid, const f4 (&r)[NQ]) {
#pragma unroll
    for (int j = 0; j < NQ; ++j) *(f4*)&lds[(tid >> 4) + 16 * j][4 * (tid & 15)] = r[j];
}

// JN: 16-column blocks per wave (4: 64 x 64 per wave, 128 x 128 tiles; 2:
// 64 x 32 per wave, 128 x 64 tiles for outputs at most 64 wide).
template <int JN = 4>
__device__ __forceinline__ void mma_slice32(float (*la)[KP32], float (*lb)[KP32],
                                            f4 (&acc)[4][JN], int wm, int wn, int fr, int g) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        f4 fa[4], fb[JN];
#pragma unroll
        for (int i = 0; i < 4; ++i) fa[i] = *(const f4*)&la[wm * 64 + 16 * i + fr][16 * g + 4 * c];
#pragma unroll
        for (int j = 0; j < JN; ++j)
            fb[j] = *(const f4*)&lb[wn * 16 * JN + 16 * j + fr][16 * g + 4 * c];
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < JN; ++j)
                    acc[i][j] =
                        __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i][e], fb[j][e], acc[i][j], 0, 0, 0);
    }
}

// The B operand of a 128 x 64 tile: rows n0 .. n0 + 63, four quads per thread
// (quad j: row tid / 16 + 16 j, k = 4 (tid % 16) .. + 3; zeros past N or K).
struct NarrowB {
    uint32_t fixed;
    __device__ NarrowB(const Operand<kF32, true>& op, int64_t n0, int tid)
        : fixed(op.row_off(n0 + (tid >> 4))) {}
    __device__ void fetch(const Operand<kF32, true>& op, int64_t k0, int64_t k_end, int tid,
                          f4 (&r)[NQ / 2]) const {
        const int64_t k = k0 + 4 * (tid & 15);
        const uint32_t base = fixed + (k < k_end ? op.col_off(k) : kOOB);
        const uint32_t step = 16 * op.pitch;
#pragma unroll
        for (int j = 0; j < NQ / 2; ++j) r[j] = op.load(base + j * step);
    }
};

// Epilogue of a wave's 64 x 32 block (JN = 2): as tile_epilogue, with each
// lane handed two rows (8 apart) of four columns per 16-row strip; the
// epilogue's other two row slots point past M.
__device__ __forceinline__ void strip_rows_narrow(int64_t m0w, int i, int lane, int64_t M,
                                                  int64_t (&m)[4]) {
    m[0] = m0w + i * 16 + (lane >> 3);
    m[1] = m[0] + 8;
    m[2] = m[3] = M;
}

template <class Epi>
__device__ __forceinline__ void tile_epilogue_narrow(const f4 (&acc)[4][2], char* smem,
                                                     int64_t m0w, int64_t n0w, const Epi& epi,
                                                     typename Epi::pre_t pre) {
    const int lane = threadIdx.x & 63;
    float* buf = (float*)smem + (threadIdx.x >> 6) * 16 * EP;
    const int64_t n = n0w + 4 * (lane & 7);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                buf[(4 * (lane >> 4) + v) * EP + j * 16 + (lane & 15)] = acc[i][j][v];
        __syncthreads();
        int64_t m[4];
        strip_rows_narrow(m0w, i, lane, epi.M, m);
        f4 val[4];
#pragma unroll
        for (int q = 0; q < 2; ++q)
            val[q] = *(const f4*)&buf[(8 * q + (lane >> 3)) * EP + 4 * (lane & 7)];
        val[2] = val[3] = f4{0.0f, 0.0f, 0.0f, 0.0f};
        if constexpr (Epi::kStripLoads) {
            typename Epi::pre_t next{};
            if (i < 3) {
                int64_t mn[4];
                strip_rows_narrow(m0w, i + 1, lane, epi.M, mn);
                epi.load(mn, n, next);
            }
            epi.run(m, n, val, pre);
            pre = next;
        } else {
            epi.run(m, n, val, pre);
        }
        __syncthreads();
    }
}

// One output tile at (m0, n0): the sum over k in [0, K) of A(m, k) B(n, k),
// handed to epi.
template <int JN, class Epi>
__device__ __forceinline__ void tile32(const Operand<kF32, true>& a, const Operand<kF32, true>& b,
                                       int64_t m0, int64_t n0, int64_t K, const Epi& epi,
                                       char* smem) {
    using Op = Operand<kF32, true>;
    constexpr int QB = JN == 4 ? NQ : NQ / 2;  // B quads per thread
    float (*la)[KP32] = (float (*)[KP32])smem;
    float (*lb)[KP32] = (float (*)[KP32])(smem + (size_t)BM * KP32 * sizeof(float));
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int wm = wv >> 1, wn = wv & 1, fr = lane & 15, g = lane >> 4;
    const int64_t m0w = m0 + wm * 64, n0w = n0 + wn * 16 * JN;
    const int64_t nsl = (K + BK - 1) / BK;
    const Stager<Op> sa(a, m0, tid);
    using SB = typename std::conditional<JN == 4, Stager<Op>, NarrowB>::type;
    const SB sb(b, n0, tid);
    f4 ra[NQ], rb[QB];
    f4 acc[4][JN];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < JN; ++j) acc[i][j] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    typename Epi::pre_t pre{};
    int64_t mr[4];
    if constexpr (JN == 4)
        strip_rows(m0w, 0, lane, mr);
    else
        strip_rows_narrow(m0w, 0, lane, epi.M, mr);
    const int64_t ne = n0w + (JN == 4 ? 4 * (lane & 15) : 4 * (lane & 7));
    sa.fetch(a, 0, K, tid, ra);
    sb.fetch(b, 0, K, tid, rb);
    for (int64_t sl = 0; sl < nsl; ++sl) {
        store_slice32(la, tid, ra);
#pragma unroll
        for (int j = 0; j < QB; ++j) *(f4*)&lb[(tid >> 4) + 16 * j][4 * (tid & 15)] = rb[j];
        __syncthreads();
        if (sl + 1 < nsl) {
            sa.fetch(a, (sl + 1) * BK, K, tid, ra);
            sb.fetch(b, (sl + 1) * BK, K, tid, rb);
        } else {
            epi.load(mr, ne, pre);
        }
        // Keep the loads ahead of the MFMAs (see tile()).
        __builtin_amdgcn_sched_barrier(0);
        mma_slice32<JN>(la, lb, acc, wm, wn, fr, g);
        __syncthreads();
    }
    if constexpr (JN == 4)
        tile_epilogue(acc, smem, m0w, n0w, epi, pre);
    else
        tile_epilogue_narrow(acc, smem, m0w, n0w, epi, pre);
}

// Epilogues of the linear layers' products C (M x N, row-major outputs).
enum LinMode {
    kLinStore,     // y = C + bias (bias may be null); act, if given, = SiLU(y)
    kLinAcc,       // y += C
    kLinSiluGrad,  // y = C * SiLU'(aux), aux laid out as y
};

template <int MODE>
struct LinEpi {
    static constexpr bool kOwnStore = false;
    static constexpr bool kStripLoads = MODE != kLinStore;
    struct pre_t {
        f4 v[4];
    };
    float* y;
    const float* bias;
    float* act;
    const float* aux;
    int64_t M, N;
    __device__ void load(const int64_t (&m)[4], int64_t n, pre_t& pre) const {
        if constexpr (MODE == kLinStore) {
            const ElemReader<float> rb(bias, N);
#pragma unroll
            for (int c = 0; c < 4; ++c) pre.v[0][c] = rb(n + c < N ? n + c : -1);
        } else {
            const __amdgpu_buffer_rsrc_t r =
                resource(MODE == kLinAcc ? y : aux, (uint32_t)(M * N * 4));
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t off = (n < N && m[q] < M) ? (uint32_t)((m[q] * N + n) * 4) : kOOB;
                const u4v w = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
                pre.v[q] = f4{__uint_as_float(w.x), __uint_as_float(w.y), __uint_as_float(w.z),
                              __uint_as_float(w.w)};
            }
        }
    }
    __device__ void run(const int64_t (&m)[4], int64_t n, const f4 (&v)[4],
                        const pre_t& pre) const {
        if (n >= N) return;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if (m[q] >= M) continue;
            f4 r;
            if constexpr (MODE == kLinStore) {
                r = v[q] + pre.v[0];
                if (act) {
                    f4 sv;
#pragma unroll
                    for (int c = 0; c < 4; ++c) sv[c] = r[c] * sigmoid(r[c]);
                    *(f4*)(act + m[q] * N + n) = sv;
                }
            } else if constexpr (MODE == kLinAcc) {
                r = pre.v[q] + v[q];
            } else {
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const float x = pre.v[q][c], sg = sigmoid(x);
                    r[c] = v[q][c] * (sg * fmaf(x, 1.0f - sg, 1.0f));
                }
            }
            *(f4*)(y + m[q] * N + n) = r;
        }
    }
};

// Y[M][N] (epilogue MODE) of C = A B^T: A[M][K], B[N][K], both row-major.
// JN = 2 (N <= 64): 128 x 64 tiles, so that no half-empty 128-column tile is
// multiplied.
template <int MODE, int JN = 4>
__global__ __launch_bounds__(256, 2) void linear32_kernel(const float* a, const float* b,
                                                          LinEpi<MODE> epi, int64_t K) {
    constexpr size_t kLds = (size_t)(BM + 32 * JN) * KP32 * sizeof(float);
    __shared__ __attribute__((aligned(16))) char smem[kLds > kEpiBytes ? kLds : kEpiBytes];
    const int64_t M = epi.M, N = epi.N;
    constexpr int kBNt = 32 * JN;
    const int64_t ntn = (N + kBNt - 1) / kBNt;
    const int64_t t = xcd_tile(((M + BM - 1) / BM) * ntn);
    if (t < 0) return;
    const Operand<kF32, true> oa{resource(a, (uint32_t)(M * K * 4)), (uint32_t)(K * 4), 0, 0, 0};
    const Operand<kF32, true> ob{resource(b, (uint32_t)(N * K * 4)), (uint32_t)(K * 4), 0, 0, 0};
    tile32<JN>(oa, ob, (t / ntn) * BM, (t % ntn) * kBNt, K, epi, smem);
}

// The same products for K <= KS * BK, in persistent workgroups: the grid is
// a fixed number of workgroups (a multiple of the column tiles); workgroup w
// keeps the KS B slices of column tile w % ntn in LDS for the whole launch
// and walks row tiles w / ntn, + G / ntn, ..., each A slice fetched into
// registers during the previous slice's MFMAs (the next tile's first slice
// during the current tile's last slice and epilogue), so that a tile's
// loads, products and stores overlap those of its neighbours.  Each tile's
// arithmetic is that of linear32_kernel (same fragments, same slice order),
// so the results are the same bit for bit.  Two workgroups per CU while the
// B slices take at most 128 LDS rows (KS = 1 at 128 columns, KS <= 2 at 64).
template <int JN, int KS>
constexpr int lin32p_occupancy() { return KS * 32 * JN <= 128 ? 2 : 1; }

template <int MODE, int JN, int KS>
__global__ __launch_bounds__(256, (lin32p_occupancy<JN, KS>())) void linear32p_kernel(
    const float* a, const float* b, LinEpi<MODE> epi, int64_t K) {
    constexpr int kBNt = 32 * JN;
    constexpr int QB = JN == 4 ? NQ : NQ / 2;  // B quads per thread
    // A slice (also the epilogue's strips), then the resident B slices.
    constexpr size_t kA = (size_t)BM * KP32 * sizeof(float);
    constexpr size_t kAreg = kA > kEpiBytes ? kA : kEpiBytes;
    __shared__ __attribute__((aligned(16))) char
        smem[kAreg + (size_t)KS * kBNt * KP32 * sizeof(float)];
    using Op = Operand<kF32, true>;
    const int64_t M = epi.M, N = epi.N;
    const int64_t ntn = (N + kBNt - 1) / kBNt, ntm = (M + BM - 1) / BM;
    const int64_t cn = blockIdx.x % ntn, stride = gridDim.x / ntn;
    int64_t tm = blockIdx.x / ntn;
    if (tm >= ntm) return;
    float (*la)[KP32] = (float (*)[KP32])smem;
    float (*lb)[KP32] = (float (*)[KP32])(smem + kAreg);
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int wm = wv >> 1, wn = wv & 1, fr = lane & 15, g = lane >> 4;
    const Op oa{resource(a, (uint32_t)(M * K * 4)), (uint32_t)(K * 4), 0, 0, 0};
    const Op ob{resource(b, (uint32_t)(N * K * 4)), (uint32_t)(K * 4), 0, 0, 0};
    const int64_t n0 = cn * kBNt, n0w = n0 + wn * 16 * JN;
    const int64_t ne = n0w + (JN == 4 ? 4 * (lane & 15) : 4 * (lane & 7));
    {
        using SB = typename std::conditional<JN == 4, Stager<Op>, NarrowB>::type;
        const SB sb(ob, n0, tid);
#pragma unroll
        for (int sl = 0; sl < KS; ++sl) {
            f4 rb[QB];
            sb.fetch(ob, sl * BK, K, tid, rb);
#pragma unroll
            for (int j = 0; j < QB; ++j)
                *(f4*)&lb[sl * kBNt + (tid >> 4) + 16 * j][4 * (tid & 15)] = rb[j];
        }
    }
    f4 ra[NQ];
    Stager<Op>(oa, tm * BM, tid).fetch(oa, 0, K, tid, ra);
    for (;;) {
        const int64_t m0 = tm * BM, m0w = m0 + wm * 64;
        const int64_t tn = tm + stride;
        typename LinEpi<MODE>::pre_t pre{};
        int64_t mr[4];
        if constexpr (JN == 4)
            strip_rows(m0w, 0, lane, mr);
        else
            strip_rows_narrow(m0w, 0, lane, M, mr);
        f4 acc[4][JN];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < JN; ++j) acc[i][j] = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int sl = 0; sl < KS; ++sl) {
            store_slice32(la, tid, ra);
            __syncthreads();  // this slice of A and (first pass) the B slices are in LDS
            if (sl + 1 < KS)
                Stager<Op>(oa, m0, tid).fetch(oa, (sl + 1) * BK, K, tid, ra);
            else if (tn < ntm)
                Stager<Op>(oa, tn * BM, tid).fetch(oa, 0, K, tid, ra);
            if (sl + 1 == KS) epi.load(mr, ne, pre);
            __builtin_amdgcn_sched_barrier(0);
            mma_slice32<JN>(la, lb + sl * kBNt, acc, wm, wn, fr, g);
            __syncthreads();  // la is free (for the next slice or the epilogue's strips)
        }
        if constexpr (JN == 4)
            tile_epilogue(acc, smem, m0w, n0w, epi, pre);
        else
            tile_epilogue_narrow(acc, smem, m0w, n0w, epi, pre);
        tm = tn;
        if (tm >= ntm) break;
    }
}

// out[K][N] = in[N][K] (the data gradient's weight operand, once per call).
__global__ __launch_bounds__(256) void transpose_kernel(const float* in, float* out, int64_t N,
                                                        int64_t K) {
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (e >= N * K) return;
    const int64_t k = e / N, n = e % N;
    out[e] = in[n * K + k];
}

// ---- weight gradients of plain fp32 linear layers (the model around the
// BD-LRU): dW = dY^T X and db = column sums of dY, on the same tiles (3-term
// bf16 split of both operands).  Each weight gradient's error stays local to
// it; the layers' forward products and data gradients, whose errors would
// travel through the rest of the model, stay on the library's fp32 GEMMs.
// Split-M partial of dW[N][K] = sum_m dY[m][n] X[m][k]: partial[split][n][k],
// and of db[n] = sum_m dY[m][n]: dbpart[split][n].
__global__ __launch_bounds__(256, 2) void wgrad_kernel(const float* dy, const float* x,
                                                       float* partial, float* dbpart, int64_t M,
                                                       int64_t N, int64_t K, int64_t splits,
                                                       int64_t rows_per_split) {
    // A(n, m) = dY[m][n], B(k, m) = X[m][k]: memory rows are the contracted
    // index for both.
    using OpA = Operand<kF32, false>;
    using OpB = Operand<kF32, false>;
    __shared__ __attribute__((aligned(16))) char smem[lds_bytes<OpA::kPlanes, OpB::kPlanes>()];
    __shared__ float colsum[BM];
    const int64_t nto = (N + BM - 1) / BM, ntk = (K + BN - 1) / BN;
    const int64_t t = xcd_tile(nto * ntk * splits);
    if (t < 0) return;
    const int64_t split = t / (nto * ntk), tl = t % (nto * ntk);
    const int64_t to = tl / ntk, tk = tl % ntk;
    const int64_t k_begin = split * rows_per_split;
    const int64_t k_end = k_begin + rows_per_split < M ? k_begin + rows_per_split : M;
    const OpA oa{resource(dy, (uint32_t)(M * N * 4)), (uint32_t)(N * 4), 0, 0, 0};
    const OpB ob{resource(x, (uint32_t)(M * K * 4)), (uint32_t)(K * 4), 0, 0, 0};
    const DwEpi epi{partial + split * N * K, N, K};
    // The tiles of column block 0 also reduce db from the dY rows they stage.
    tile(oa, ob, to * BM, tk * BN, k_begin, k_end, epi, smem, tk == 0 ? colsum : nullptr);
    if (tk == 0) {
        const int64_t o = to * BM + threadIdx.x;
        if (threadIdx.x < BM && o < N) dbpart[split * N + o] = colsum[threadIdx.x];
    }
}

// ---- fused recurrent step with the gate projections (decode)
// One tile covers 64 channels: with the weights packed so that each wave's 64
// columns are [z_r of 32 channels | z_i of the same 32 channels], MFMA block
// j < 2 of a lane holds z_r and block j + 2 holds z_i of the same (row,
// channel), and the step h_next = alpha h_prev + beta x runs on the
// accumulators directly: z never leaves the registers.
// Packed row n (of ceil(D / 64) * 128): channel block n / 128, wave half
// w = (n / 64) % 2, gate (n / 32) % 2, channel (n / 128) * 64 + 32 w + n % 32.
__host__ __device__ inline int64_t step_pack_rows(int64_t D) { return (D + 63) / 64 * 128; }

template <typename T>
__global__ __launch_bounds__(256) void pack_step_kernel(const T* wr, const T* wi, __bf16* out,
                                                        int64_t D) {
    const int64_t rows = step_pack_rows(D), total = rows * D;
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= total) return;
    const int64_t n = e / D, k = e % D;
    const int64_t ch = (n / 128) * 64 + 32 * ((n / 64) % 2) + n % 32;
    const bool gate_i = (n / 32) % 2 == 1;
    float v = 0.0f;
    if (ch < D) v = gate_i ? to_f32(wi[ch * D + k]) : to_f32(wr[ch * D + k]);
    const __bf16 hi = (__bf16)v;
    out[e] = hi;
    if (sizeof(T) == 4) out[total + e] = (__bf16)(v - (float)hi);
}

template <typename T>
struct StepEpi {
    static constexpr bool kOwnStore = true;
    static constexpr bool kStripLoads = false;
    // Everything the step reads besides z, for the lane's 2 x 4 x 4 elements
    // (channel block j, strip i, row v): loaded before any store.
    struct pre_t {
        float x[2][4][4], hp[2][4][4];
        ChannelConst cc[2];
        float bzr[2], bzi[2];
    };
    const T* x;
    const T* br;
    const T* bi;
    const float* lam;
    const float* h_prev;
    float* h_next;
    int64_t B, D;
    // m[0] is the lane's first row of strip 0; n is the tile column of the
    // lane's first output (n0w + 4 (lane % 16)), unused here.
    __device__ void load(const int64_t (&m)[4], int64_t, pre_t& pre) const {
        const int lane = threadIdx.x & 63;
        const int64_t m0w = m[0] - (lane >> 4);
        const int64_t ch0 = chan0();
        const ElemReader<T> rx(x, B * D), rbr(br, D), rbi(bi, D);
        const ElemReader<float> rh(h_prev, B * D), rl(lam, D);
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int64_t ch = ch0 + 16 * j;
            const bool okc = ch < D;
            pre.cc[j] = channel_const(rl(okc ? ch : -1));
            pre.bzr[j] = rbr(okc ? ch : -1);
            pre.bzi[j] = rbi(okc ? ch : -1);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int64_t b = m0w + i * 16 + 4 * (lane >> 4) + v;
                    const int64_t e = (okc && b < B) ? b * D + ch : -1;
                    pre.x[j][i][v] = rx(e);
                    pre.hp[j][i][v] = rh(e);
                }
        }
    }
    __device__ int64_t chan0() const { return ch_base + (threadIdx.x & 15); }
    int64_t ch_base = 0;  // first channel of this wave's 32 (set per tile)
    __device__ void store_tile(const f4 (&acc)[4][4], int64_t m0w, int64_t, const pre_t& pre) const {
        const int lane = threadIdx.x & 63;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int64_t ch = chan0() + 16 * j;
            if (ch >= D) continue;
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int64_t b = m0w + i * 16 + 4 * (lane >> 4) + v;
                    if (b >= B) continue;
                    float a, u;
                    gate_forward(pre.x[j][i][v], acc[i][j][v] + pre.bzr[j],
                                 acc[i][j + 2][v] + pre.bzi[j], pre.cc[j], a, u);
                    h_next[b * D + ch] = fmaf(a, pre.hp[j][i][v], u);
                }
        }
    }
};

// One tile of 128 batch rows x 64 channels per workgroup; pack holds the
// step-ordered weight planes.  h_next may equal h_prev.
template <typename T>
__global__ __launch_bounds__(256, 2) void step_kernel(const T* x, const __bf16* pack,
                                                      const T* br, const T* bi, const float* lam,
                                                      const float* h_prev, float* h_next,
                                                      int64_t B, int64_t D) {
    constexpr bool F32 = sizeof(T) == 4;
    using OpA = Operand<F32 ? kF32 : kBf16, true>;
    using OpB = Operand<F32 ? kPack2 : kPack1, true>;
    __shared__ __attribute__((aligned(16))) char smem[lds_bytes<OpA::kPlanes, OpB::kPlanes>()];
    const int64_t ntn = step_pack_rows(D) / BN;
    const int64_t t = xcd_tile(((B + BM - 1) / BM) * ntn);
    if (t < 0) return;
    const uint32_t plane = (uint32_t)(step_pack_rows(D) * D * 2);
    const OpA a{resource(x, (uint32_t)(B * D * sizeof(T))), (uint32_t)(D * sizeof(T)), 0, 0, 0};
    const OpB b{resource(pack, OpB::kPlanes * plane), (uint32_t)(D * 2), 0, 0, plane};
    StepEpi<T> epi{x, br, bi, lam, h_prev, h_next, B, D};
    // Columns n0w.. of wave half wn hold channels (n0w / 2).. (see the packing).
    epi.ch_base = ((t % ntn) * BN + ((threadIdx.x >> 6) & 1) * 64) / 2;
    tile(a, b, (t / ntn) * BM, (t % ntn) * BN, 0, D, epi, smem);
}

// Sums the split-K partials (fp64) in a fixed order: block column g of 8 sums
// its contiguous run of splits in ascending order, then the 8 runs are added
// in order.  64 consecutive outputs per workgroup keep the reads coalesced.
constexpr int kRedGroups = 8;
__global__ __launch_bounds__(64 * kRedGroups) void dw_reduce_kernel(
    const float* partial, const float* dbpart, int64_t splits, int64_t D, float* dwr, float* dbr,
    float* dwi, float* dbi) {
    const int64_t total = 2 * D * D;
    const int el = threadIdx.x & 63, g = threadIdx.x >> 6;
    const int64_t e = (int64_t)blockIdx.x * 64 + el;
    const int64_t per = (splits + kRedGroups - 1) / kRedGroups;
    const int64_t s0 = g * per;
    const int64_t s1 = s0 + per < splits ? s0 + per : splits;
    double s = 0.0;
    if (e < total + 2 * D) {
        const float* src = e < total ? partial + e : dbpart + (e - total);
        const int64_t stride = e < total ? total : 2 * D;
#pragma unroll 8
        for (int64_t k = s0; k < s1; ++k) s += (double)src[k * stride];
    }
    __shared__ double red[kRedGroups][64];
    red[g][el] = s;
    __syncthreads();
    if (g != 0 || e >= total + 2 * D) return;
    double t = red[0][el];
#pragma unroll
    for (int gg = 1; gg < kRedGroups; ++gg) t += red[gg][el];
    if (e < total) {
        const int64_t o = e / D, c = e % D;
        if (o < D) dwr[o * D + c] = (float)t;
        else dwi[(o - D) * D + c] = (float)t;
    } else {
        const int64_t o = e - total;
        if (o < D) dbr[o] = (float)t;
        else dbi[o - D] = (float)t;
    }
}

// Split count and rows per split (a multiple of BK) of the weight gradient:
// about two workgroups per CU, at least 512 rows per split.
void dw_split(int64_t M, int64_t D, int64_t* splits, int64_t* rows) {
    const int64_t tiles = ((2 * D + BM - 1) / BM) * ((D + BN - 1) / BN);
    int64_t s = 512 / tiles;
    const int64_t by_rows = (M + 511) / 512;
    if (s > by_rows) s = by_rows;
    if (s < 1) s = 1;
    int64_t r = (M + s - 1) / s;
    r = (r + BK - 1) / BK * BK;
    if (r < BK) r = BK;
    *rows = r;
    *splits = (M + r - 1) / r;
    if (*splits < 1) *splits = 1;
}

}  // namespace fastmm

namespace {
constexpr int64_t kFastLimit = (int64_t)1 << 31;  // bytes addressable by one buffer resource here

bool aligned16(std::initializer_list<const void*> ptrs) {
    for (const void* p : ptrs)
        if ((uintptr_t)p % 16 != 0) return false;
    return true;
}

// Byte distance from lo to hi if the pair [lo, lo + n) and [hi, hi + n) can
// be addressed as one resource (hi after lo, 16-byte steps), else -1.
int64_t pair_offset(const void* lo, const void* hi, int64_t n_bytes, int64_t tail_bytes) {
    const int64_t d = (const char*)hi - (const char*)lo;
    if (d < n_bytes || d % 16 != 0) return -1;
    return d + n_bytes + tail_bytes < kFastLimit ? d : -1;
}
}  // namespace

// ------------------------------------------------------------------ launchers
static dim3 tiles(int64_t M, int64_t N, int64_t z = 1) {
    return dim3((unsigned)((M + kTM - 1) / kTM), (unsigned)((N + kTN - 1) / kTN), (unsigned)z);
}

size_t project_pack_workspace(int64_t D, IoType io) {
    return (size_t)(io == IoType::kF32 ? 2 : 1) * (size_t)(2 * D * D) * 2;
}

static hipError_t launch_pack(const void* wr, const void* wi, int64_t D, IoType io,
                              bool transposed, void* pack, hipStream_t stream) {
    const dim3 grid((unsigned)((2 * D * D + 255) / 256));
    if (io == IoType::kF32) {
        if (transposed)
            hipLaunchKernelGGL((fastmm::pack_kernel<float, true>), grid, dim3(256), 0, stream,
                               (const float*)wr, (const float*)wi, (__bf16*)pack, D);
        else
            hipLaunchKernelGGL((fastmm::pack_kernel<float, false>), grid, dim3(256), 0, stream,
                               (const float*)wr, (const float*)wi, (__bf16*)pack, D);
    } else {
        if (transposed)
            hipLaunchKernelGGL((fastmm::pack_kernel<bf16, true>), grid, dim3(256), 0, stream,
                               (const bf16*)wr, (const bf16*)wi, (__bf16*)pack, D);
        else
            hipLaunchKernelGGL((fastmm::pack_kernel<bf16, false>), grid, dim3(256), 0, stream,
                               (const bf16*)wr, (const bf16*)wi, (__bf16*)pack, D);
    }
    return hipGetLastError();
}

hipError_t launch_project_forward(const void* x, const void* wr, const void* br, const void* wi,
                                  const void* bi, void* zr, void* zi, int64_t M, int64_t D,
                                  IoType io, void* pack, hipStream_t stream) {
    if (M == 0 || D == 0) return hipSuccess;
    const int64_t esz = io == IoType::kF32 ? 4 : 2;
    if (D % 8 == 0 && aligned16({x, zr, zi, pack}) &&
        (M + fastmm::BM) * D * esz < kFastLimit) {
        hipError_t e = launch_pack(wr, wi, D, io, false, pack, stream);
        if (e != hipSuccess) return e;
        const int64_t tiles = ((M + fastmm::BM - 1) / fastmm::BM) *
                              ((2 * D + fastmm::BN - 1) / fastmm::BN);
        if (io == IoType::kF32)
            hipLaunchKernelGGL(fastmm::fwd_kernel<float>, dim3(fastmm::grid_of(tiles)), dim3(256),
                               0, stream, (const float*)x, (const __bf16*)pack, (const float*)br,
                               (const float*)bi, (float*)zr, (float*)zi, M, D);
        else
            hipLaunchKernelGGL(fastmm::fwd_kernel<bf16>, dim3(fastmm::grid_of(tiles)), dim3(256),
                               0, stream, (const bf16*)x, (const __bf16*)pack, (const bf16*)br,
                               (const bf16*)bi, (float*)zr, (float*)zi, M, D);
        return hipGetLastError();
    }
    if (io == IoType::kF32)
        hipLaunchKernelGGL(proj_fwd_kernel<float>, tiles(M, 2 * D), dim3(kThreads), 0, stream,
                           (const float*)x, (const float*)wr, (const float*)br,
                           (const float*)wi, (const float*)bi, (float*)zr, (float*)zi, M, D);
    else
        hipLaunchKernelGGL(proj_fwd_kernel<bf16>, tiles(M, 2 * D), dim3(kThreads), 0, stream,
                           (const bf16*)x, (const bf16*)wr, (const bf16*)br, (const bf16*)wi,
                           (const bf16*)bi, (float*)zr, (float*)zi, M, D);
    return hipGetLastError();
}

hipError_t launch_project_backward_data(const void* dzr, const void* dzi, const void* wr,
                                        const void* wi, void* dx, int64_t M, int64_t D,
                                        IoType io, void* pack, hipStream_t stream, bool dx_f32) {
    if (M == 0 || D == 0) return hipSuccess;
    dx_f32 = dx_f32 && io == IoType::kBf16;
    const int64_t hoff = pair_offset(dzr, dzi, M * D * 4, fastmm::BM * D * 4);
    if (D % 8 == 0 && hoff >= 0 && aligned16({dzr, dx, pack})) {
        hipError_t e = launch_pack(wr, wi, D, io, true, pack, stream);
        if (e != hipSuccess) return e;
        const int64_t tiles = ((M + fastmm::BM - 1) / fastmm::BM) *
                              ((D + fastmm::BN - 1) / fastmm::BN);
        if (io == IoType::kF32)
            hipLaunchKernelGGL(fastmm::dx_kernel<float>, dim3(fastmm::grid_of(tiles)), dim3(256),
                               0, stream, (const float*)dzr, (uint32_t)hoff, (const __bf16*)pack,
                               (float*)dx, M, D);
        else if (dx_f32)
            hipLaunchKernelGGL((fastmm::dx_kernel<bf16, float>), dim3(fastmm::grid_of(tiles)),
                               dim3(256), 0, stream, (const float*)dzr, (uint32_t)hoff,
                               (const __bf16*)pack, (float*)dx, M, D);
        else
            hipLaunchKernelGGL(fastmm::dx_kernel<bf16>, dim3(fastmm::grid_of(tiles)), dim3(256),
                               0, stream, (const float*)dzr, (uint32_t)hoff, (const __bf16*)pack,
                               (bf16*)dx, M, D);
        return hipGetLastError();
    }
    if (io == IoType::kF32)
        hipLaunchKernelGGL(proj_dx_kernel<float>, tiles(M, D), dim3(kThreads), 0, stream,
                           (const float*)dzr, (const float*)dzi, (const float*)wr,
                           (const float*)wi, (float*)dx, M, D);
    else if (dx_f32)
        hipLaunchKernelGGL((proj_dx_kernel<bf16, float>), tiles(M, D), dim3(kThreads), 0, stream,
                           (const float*)dzr, (const float*)dzi, (const bf16*)wr, (const bf16*)wi,
                           (float*)dx, M, D);
    else
        hipLaunchKernelGGL(proj_dx_kernel<bf16>, tiles(M, D), dim3(kThreads), 0, stream,
                           (const float*)dzr, (const float*)dzi, (const bf16*)wr, (const bf16*)wi,
                           (bf16*)dx, M, D);
    return hipGetLastError();
}

hipError_t launch_pack_groups(const void* wr, const void* wi, int64_t D, IoType io, void* pack,
                              hipStream_t stream) {
    const dim3 grid((unsigned)((2 * D * D + 255) / 256));
    if (io == IoType::kF32)
        hipLaunchKernelGGL(fastmm::pack_group_kernel<float>, grid, dim3(256), 0, stream,
                           (const float*)wr, (const float*)wi, (__bf16*)pack, D);
    else
        hipLaunchKernelGGL(fastmm::pack_group_kernel<bf16>, grid, dim3(256), 0, stream,
                           (const bf16*)wr, (const bf16*)wi, (__bf16*)pack, D);
    return hipGetLastError();
}

size_t step_pack_workspace(int64_t D, IoType io) {
    return (size_t)(io == IoType::kF32 ? 2 : 1) * (size_t)(fastmm::step_pack_rows(D) * D) * 2;
}

bool launch_fused_step(const void* x, const void* wr, const void* br, const void* wi,
                       const void* bi, const float* lambda, const float* h_prev, float* h_next,
                       int64_t B, int64_t D, IoType io, void* pack, hipStream_t stream,
                       hipError_t* err) {
    const int64_t esz = io == IoType::kF32 ? 4 : 2;
    if (B == 0 || D % 8 != 0 || !aligned16({x, pack}) || (B + fastmm::BM) * D * esz >= kFastLimit)
        return false;
    const int64_t rows = fastmm::step_pack_rows(D);
    const dim3 pgrid((unsigned)((rows * D + 255) / 256));
    const int64_t tiles = ((B + fastmm::BM - 1) / fastmm::BM) * (rows / fastmm::BN);
    if (io == IoType::kF32) {
        hipLaunchKernelGGL(fastmm::pack_step_kernel<float>, pgrid, dim3(256), 0, stream,
                           (const float*)wr, (const float*)wi, (__bf16*)pack, D);
        hipLaunchKernelGGL(fastmm::step_kernel<float>, dim3(fastmm::grid_of(tiles)), dim3(256), 0,
                           stream, (const float*)x, (const __bf16*)pack, (const float*)br,
                           (const float*)bi, lambda, h_prev, h_next, B, D);
    } else {
        hipLaunchKernelGGL(fastmm::pack_step_kernel<bf16>, pgrid, dim3(256), 0, stream,
                           (const bf16*)wr, (const bf16*)wi, (__bf16*)pack, D);
        hipLaunchKernelGGL(fastmm::step_kernel<bf16>, dim3(fastmm::grid_of(tiles)), dim3(256), 0,
                           stream, (const bf16*)x, (const __bf16*)pack, (const bf16*)br,
                           (const bf16*)bi, lambda, h_prev, h_next, B, D);
    }
    *err = hipGetLastError();
    return true;
}

int64_t project_dw_splits(int64_t M, int64_t D) {
    // Enough workgroups to fill the GPU: aim for ~1024 tiles in total.
    int64_t tiles_per_split = ((2 * D + kTM - 1) / kTM) * ((D + 1 + kTN - 1) / kTN);
    int64_t splits = 1024 / (tiles_per_split > 0 ? tiles_per_split : 1);
    if (splits < 1) splits = 1;
    int64_t max_by_rows = (M + 255) / 256;  // at least 256 rows per split
    if (splits > max_by_rows) splits = max_by_rows;
    if (splits < 1) splits = 1;
    return splits;
}

size_t project_dw_workspace(int64_t M, int64_t D) {
    // Either path may run (the choice depends on pointer alignment): size for both.
    const size_t generic =
        (size_t)project_dw_splits(M, D) * (size_t)(2 * D) * (size_t)(D + 1) * sizeof(float);
    int64_t splits = 1, rows = 0;
    fastmm::dw_split(M, D, &splits, &rows);
    const size_t fast = (size_t)splits * (size_t)(2 * D) * (size_t)(D + 1) * sizeof(float);
    return generic > fast ? generic : fast;
}

hipError_t launch_project_backward_weights(const void* dzr, const void* dzi, const void* x,
                                           float* dwr, float* dbr, float* dwi, float* dbi,
                                           int64_t M, int64_t D, IoType io, void* ws,
                                           hipStream_t stream) {
    if (D == 0) return hipSuccess;
    const int64_t esz = io == IoType::kF32 ? 4 : 2;
    const int64_t hoff = pair_offset(dzr, dzi, M * D * 4, fastmm::BK * D * 4);
    if (D % 8 == 0 && M > 0 && hoff >= 0 && aligned16({dzr, x, ws}) &&
        (M + fastmm::BK) * D * esz < kFastLimit) {
        int64_t splits = 1, rows_per_split = 0;
        fastmm::dw_split(M, D, &splits, &rows_per_split);
        const int64_t tiles = ((2 * D + fastmm::BM - 1) / fastmm::BM) *
                              ((D + fastmm::BN - 1) / fastmm::BN) * splits;
        float* partial = (float*)ws;
        float* dbpart = partial + splits * 2 * D * D;
        if (io == IoType::kF32)
            hipLaunchKernelGGL(fastmm::dw_kernel<float>, dim3(fastmm::grid_of(tiles)), dim3(256),
                               0, stream, (const float*)dzr, (uint32_t)hoff, (const float*)x,
                               partial, dbpart, M, D, splits, rows_per_split);
        else
            hipLaunchKernelGGL(fastmm::dw_kernel<bf16>, dim3(fastmm::grid_of(tiles)), dim3(256),
                               0, stream, (const float*)dzr, (uint32_t)hoff, (const bf16*)x,
                               partial, dbpart, M, D, splits, rows_per_split);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        const int64_t total = 2 * D * D + 2 * D;
        hipLaunchKernelGGL(fastmm::dw_reduce_kernel, dim3((unsigned)((total + 63) / 64)),
                           dim3(64 * fastmm::kRedGroups), 0, stream, (const float*)partial,
                           (const float*)dbpart, splits, D, dwr, dbr, dwi, dbi);
        return hipGetLastError();
    }
    const int64_t splits = project_dw_splits(M, D);
    const int64_t rows_per_split = (M + splits - 1) / splits;
    float* partial = (float*)ws;
    if (io == IoType::kF32)
        hipLaunchKernelGGL(proj_dw_kernel<float>, tiles(2 * D, D + 1, splits), dim3(kThreads), 0,
                           stream, (const float*)dzr, (const float*)dzi, (const float*)x, partial,
                           M, D, rows_per_split);
    else
        hipLaunchKernelGGL(proj_dw_kernel<bf16>, tiles(2 * D, D + 1, splits), dim3(kThreads), 0,
                           stream, (const float*)dzr, (const float*)dzi, (const bf16*)x, partial,
                           M, D, rows_per_split);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t total = 2 * D * (D + 1);
    hipLaunchKernelGGL(proj_dw_reduce_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0,
                       stream, (const float*)partial, splits, D, dwr, dbr, dwi, dbi);
    return hipGetLastError();
}

// ------------------------------------------------------------------ linear layers
bool wgrad_fast_ok(std::initializer_list<const void*> ptrs, int64_t M, int64_t N, int64_t K) {
    return M > 0 && N > 0 && K > 0 && N % 4 == 0 && K % 4 == 0 && aligned16(ptrs) &&
           (M + fastmm::BM) * (N > K ? N : K) * 4 < kFastLimit;
}

namespace {
// Tiles of a linear-layer product with output width N: 128 x 64 when N <= 64.
int64_t linear_tiles(int64_t M, int64_t N) {
    const int64_t bn = N <= 64 ? 64 : fastmm::BN;
    return ((M + fastmm::BM - 1) / fastmm::BM) * ((N + bn - 1) / bn);
}
// Compute units of the current device (256 if the query fails).
int device_cus() {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus < 1)
        cus = 256;
    return cus;
}

template <int MODE>
void launch_lin32(const float* a, const float* b, const fastmm::LinEpi<MODE>& e, int64_t K,
                  hipStream_t stream) {
    const dim3 block(256);
    const int64_t tiles = linear_tiles(e.M, e.N);
    // Persistent workgroups where the B slices stay in LDS: K <= 64, or
    // K <= 128 with outputs at most 64 wide.
    // (At K = 256 four slices in LDS need one workgroup per CU, 159-162
    // against 147-155 us on the tile kernel; the B fragments held in
    // registers instead, 128 VGPRs per wave, spill and measured 143-163
    // against 149-157 us; one 8-wave workgroup whose two halves share the
    // resident slices and walk alternate row tiles, 158-179 against
    // 148-157 us: the halves run in lockstep and do not overlap.)
    const int ks = K <= fastmm::BK ? 1 : (K <= 2 * fastmm::BK && e.N <= 64 ? 2 : 0);
    if (ks > 0) {
        const int64_t ntn = tiles / ((e.M + fastmm::BM - 1) / fastmm::BM);
        int64_t g = 2 * (int64_t)device_cus();
        g = g / ntn * ntn;
        if (g > tiles) g = tiles;
        if (g < ntn) g = ntn;
        const dim3 grid((unsigned)g);
        if (e.N <= 64 && ks == 2)
            hipLaunchKernelGGL((fastmm::linear32p_kernel<MODE, 2, 2>), grid, block, 0, stream, a, b, e, K);
        else if (e.N <= 64)
            hipLaunchKernelGGL((fastmm::linear32p_kernel<MODE, 2, 1>), grid, block, 0, stream, a, b, e, K);
        else
            hipLaunchKernelGGL((fastmm::linear32p_kernel<MODE, 4, 1>), grid, block, 0, stream, a, b, e, K);
        return;
    }
    const dim3 grid(fastmm::grid_of(tiles));
    if (e.N <= 64)
        hipLaunchKernelGGL((fastmm::linear32_kernel<MODE, 2>), grid, block, 0, stream, a, b, e, K);
    else
        hipLaunchKernelGGL((fastmm::linear32_kernel<MODE, 4>), grid, block, 0, stream, a, b, e, K);
}
}  // namespace

hipError_t launch_linear_fwd32(const float* x, const float* w, const float* bias, float* y,
                               float* act, int64_t M, int64_t N, int64_t K, hipStream_t stream) {
    const fastmm::LinEpi<fastmm::kLinStore> e{y, bias, act, nullptr, M, N};
    launch_lin32(x, w, e, K, stream);
    return hipGetLastError();
}

hipError_t launch_linear_dgrad32(const float* dy, const float* w, float* dx, LinearMode mode,
                                 const float* aux, int64_t M, int64_t N, int64_t K, float* wt,
                                 hipStream_t stream) {
    hipLaunchKernelGGL(fastmm::transpose_kernel, dim3((unsigned)((N * K + 255) / 256)), dim3(256),
                       0, stream, w, wt, N, K);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    // dX[M][K] = dY[M][N] W^T[K][N]^T: output width K, contraction N.
    switch (mode) {
        case LinearMode::kStore:
            launch_lin32(dy, wt, fastmm::LinEpi<fastmm::kLinStore>{dx, nullptr, nullptr, nullptr, M, K},
                         N, stream);
            break;
        case LinearMode::kAccumulate:
            launch_lin32(dy, wt, fastmm::LinEpi<fastmm::kLinAcc>{dx, nullptr, nullptr, nullptr, M, K},
                         N, stream);
            break;
        case LinearMode::kSiluGrad:
            launch_lin32(dy, wt, fastmm::LinEpi<fastmm::kLinSiluGrad>{dx, nullptr, nullptr, aux, M, K},
                         N, stream);
            break;
    }
    return hipGetLastError();
}

// About one workgroup per CU in all (each split's partial is summed again
// afterwards: on the model step, 256 workgroups measured 11.8 ms, 512
// 12.0 ms and 1024 12.2 ms), at least 256 rows per split.
int64_t wgrad_splits(int64_t M, int64_t N, int64_t K) {
    const int64_t t = ((N + fastmm::BM - 1) / fastmm::BM) * ((K + fastmm::BN - 1) / fastmm::BN);
    int64_t s = 256 / t;
    const int64_t by_rows = (M + 255) / 256;
    if (s > by_rows) s = by_rows;
    return s < 1 ? 1 : s;
}

size_t wgrad_workspace(int64_t M, int64_t N, int64_t K) {
    return (size_t)wgrad_splits(M, N, K) * (size_t)(N * K + N) * sizeof(float);
}

hipError_t launch_wgrad(const float* dy, const float* x, float* dw, float* db, int64_t M,
                        int64_t N, int64_t K, void* ws, void* colsum_ws, hipStream_t stream) {
    const int64_t splits = wgrad_splits(M, N, K);
    const int64_t rows = (M + splits - 1) / splits;
    float* partial = (float*)ws;
    float* dbpart = partial + splits * N * K;
    const int64_t t = splits * ((N + fastmm::BM - 1) / fastmm::BM) *
                      ((K + fastmm::BN - 1) / fastmm::BN);
    hipLaunchKernelGGL(fastmm::wgrad_kernel, dim3(fastmm::grid_of(t)), dim3(256), 0, stream, dy,
                       x, partial, dbpart, M, N, K, splits, rows);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = launch_colsum(partial, splits, N * K, dw, colsum_ws, stream);
    if (e != hipSuccess || !db) return e;
    return launch_colsum(dbpart, splits, N, db, colsum_ws, stream);
}

}  // namespace recblr
