// Gate projections of the BD-LRU (RecBLR, arXiv 2406.12580, section 3.2):
//   z_r = x W_r^T + b_r,  z_i = x W_i^T + b_i            (forward)
//   dx += dz_r W_r + dz_i W_i                            (backward, data)
//   dW_r = dz_r^T x, dW_i = dz_i^T x, db = sum_rows dz   (backward, weights)
// One tiled kernel serves all three products through operand accessors; the
// two gates are handled as one concatenated operand of width 2D.  x and the
// weights use the I/O type; z and dz are fp32 scratch (rounding them to bf16
// would cost about 1e-2 of relative accuracy in dW).
//
// Tiling: a 256-thread workgroup (4 waves) computes a 64 x 64 tile of C = A B
// on the matrix cores; each wave owns a 32 x 32 quarter as 2 x 2 MFMA blocks of
// 16 x 16 (v_mfma_f32_16x16x4_f32, or v_mfma_f32_16x16x32_bf16 when both
// operands are bf16 inputs), accumulating in fp32.  K-slices of A and B are
// staged through LDS in a K-contiguous layout; each operand is read from
// global memory in the order that is contiguous for it.  The weight-gradient
// product reduces over all B*L rows and is split across workgroups
// (split-K); its fp32 partial tiles are summed afterwards in a fixed order,
// so results are deterministic.
#include <initializer_list>
#include <type_traits>

#include "device_common.hpp"
#include "gemm.hpp"

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

template <typename T>
__global__ __launch_bounds__(kThreads) void proj_dx_kernel(const float* dzr, const float* dzi,
                                                           const T* wr, const T* wi, T* dx,
                                                           int64_t M, int64_t D) {
    DxOps<T> ops{dzr, dzi, wr, wi, D};
    mfma_tile<false>(ops, M, D, 0, 2 * D, [&](int64_t i, int64_t n, float v) {
        T* p = dx + i * D + n;
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
// Taken when D % 8 == 0 and the operands are 16-byte aligned (every workload
// shape of the paper).  A 256-thread workgroup computes a 128 x 128 tile of
// C = A B; each wave owns a 64 x 64 quarter as 4 x 4 blocks of
// v_mfma_f32_16x16x32_bf16.  An fp32 operand is split on load into
// hi = bf16(v) and lo = bf16(v - hi) and the product is formed from the three
// terms hi*hi + hi*lo + lo*hi (a bf16 operand is exact and needs one plane):
// each product then carries a relative error below 3 * 2^-17 against 2^-24
// for a plain fp32 product, while the matrix cores deliver 16x the fp32 MFMA
// rate, so the projection stays bound by HBM instead of by fp32 MFMA.
// Operand quads (4 consecutive elements along the contiguous memory index)
// are prefetched into registers for the next K-slice while the current slice
// is multiplied from LDS.  Tiles are ordered so that consecutive tiles of one
// row block land on the same XCD and share its L2.
namespace fastmm {
#ifndef RECBLR_GEMM_BK
#define RECBLR_GEMM_BK 64
#endif
constexpr int BM = 128, BN = 128, BK = RECBLR_GEMM_BK;
static_assert(BK == 32 || BK == 64, "K-slice depth");
constexpr int NQ = BK / 8;  // quads per thread and operand in one slice
// LDS row pitch (bf16 elements): BK + 8 keeps rows 16-byte aligned and the
// fragment reads of 8 consecutive rows on distinct banks.
constexpr int KP = BK + 8;
typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f8 __attribute__((ext_vector_type(8)));
typedef __bf16 b4 __attribute__((ext_vector_type(4)));
typedef __bf16 b8 __attribute__((ext_vector_type(8)));

// A quad (4 consecutive elements) as loaded: fp32 values or raw bf16 bits.
__device__ __forceinline__ f4 raw_quad(const float* p) { return *(const f4*)p; }
__device__ __forceinline__ uint2 raw_quad(const bf16* p) { return *(const uint2*)p; }
__device__ __forceinline__ f4 widen(f4 v) { return v; }
__device__ __forceinline__ f4 widen(uint2 v) {
    return f4{__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u),
              __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xffff0000u)};
}
__device__ __forceinline__ f4 load_quad(const float* p) { return raw_quad(p); }
__device__ __forceinline__ f4 load_quad(const bf16* p) { return widen(raw_quad(p)); }
// Element c of a raw quad as 16 bf16 bits.
__device__ __forceinline__ uint32_t bits16(uint2 v, int c) {
    const uint32_t w = c < 2 ? v.x : v.y;
    return (c & 1) ? w >> 16 : w & 0xffffu;
}

// Memory views: at(row, col) points at element (row, col), contiguous along col.
template <typename T>
struct PlainMem {
    const T* p;
    int64_t ld;
    __device__ const T* at(int64_t row, int64_t col) const { return p + row * ld + col; }
};
// Rows [0, split) come from p0, the rest from p1 (both with pitch ld).
template <typename T>
struct RowPairMem {
    const T* p0;
    const T* p1;
    int64_t split, ld;
    __device__ const T* at(int64_t row, int64_t col) const {
        return row < split ? p0 + row * ld + col : p1 + (row - split) * ld + col;
    }
};
// Columns [0, split) come from p0, the rest from p1 (both with pitch split).
template <typename T>
struct ColPairMem {
    const T* p0;
    const T* p1;
    int64_t split;
    __device__ const T* at(int64_t row, int64_t col) const {
        return col < split ? p0 + row * split + col : p1 + row * split + (col - split);
    }
};

// Operand with element (mn, k): mn is the row of A (or column of B), k the
// contracted index.  KFAST: memory is contiguous along k (element at
// mem.at(mn, k)); otherwise along mn (element at mem.at(k, mn)).  mn_end is
// the number of valid mn (a multiple of 4).
template <typename T, bool KFAST, class Mem>
struct Operand {
    static constexpr bool kKFast = KFAST;
    static constexpr int kPlanes = sizeof(T) == 4 ? 2 : 1;
    using raw_t = decltype(raw_quad((const T*)nullptr));
    Mem mem;
    int64_t mn_end;
    __device__ raw_t quad(int64_t mn, int64_t k) const {
        return raw_quad(KFAST ? mem.at(mn, k) : mem.at(k, mn));
    }
};

// Staging of one operand's 128 x BK slice: NQ = BK / 8 quads per thread.
//   KFAST: quad j covers (mn = e / (BK / 4), k = 4 (e % (BK / 4)) .. +3) with e = tid + 256 j.
//   else : quad j covers (mn = 4 (tid % 32) .. +3, k = NQ (tid / 32) + j).
template <class Op>
__device__ __forceinline__ void fetch_slice(const Op& op, int64_t mn0, int64_t k0, int64_t k_end,
                                            int tid, typename Op::raw_t (&r)[NQ]) {
#pragma unroll
    for (int j = 0; j < NQ; ++j) {
        int64_t mn, k;
        if constexpr (Op::kKFast) {
            const int e = tid + 256 * j;
            mn = mn0 + e / (BK / 4);
            k = k0 + 4 * (e % (BK / 4));
        } else {
            mn = mn0 + 4 * (tid & 31);
            k = k0 + NQ * (tid >> 5) + j;
        }
        r[j] = (mn < op.mn_end && k < k_end) ? op.quad(mn, k) : typename Op::raw_t{};
    }
}

template <int N>
struct PackT;
template <>
struct PackT<4> {
    using bits = uint2;
    using fv = f4;
    using bv = b4;
};
template <>
struct PackT<8> {
    using bits = uint4;
    using fv = f8;
    using bv = b8;
};

template <class Op>
__device__ __forceinline__ void store_slice(__bf16 (*lds)[BM][KP], int tid,
                                            const typename Op::raw_t (&r)[NQ]) {
    constexpr int P = Op::kPlanes;
    if constexpr (Op::kKFast) {
#pragma unroll
        for (int j = 0; j < NQ; ++j) {
            const int e = tid + 256 * j;
            const int row = e / (BK / 4), kc = 4 * (e % (BK / 4));
            if constexpr (P == 1) {
                *(uint2*)&lds[0][row][kc] = r[j];  // bf16 input: store the bits as they are
            } else {
                const f4 v = widen(r[j]);
                const b4 hi = __builtin_convertvector(v, b4);
                *(b4*)&lds[0][row][kc] = hi;
                *(b4*)&lds[1][row][kc] =
                    __builtin_convertvector(v - __builtin_convertvector(hi, f4), b4);
            }
        }
    } else {
        // Transpose in registers: column c of the thread's quads becomes NQ
        // consecutive k of LDS row 4 mq + c.
        using PK = PackT<NQ>;
        const int mq = tid & 31, kc = NQ * (tid >> 5);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            if constexpr (P == 1) {
                uint32_t w[NQ / 2];
#pragma unroll
                for (int j = 0; j < NQ / 2; ++j)
                    w[j] = bits16(r[2 * j], c) | (bits16(r[2 * j + 1], c) << 16);
                *(typename PK::bits*)&lds[0][4 * mq + c][kc] = *(const typename PK::bits*)w;
            } else {
                typename PK::fv v;
#pragma unroll
                for (int j = 0; j < NQ; ++j) v[j] = widen(r[j])[c];
                const typename PK::bv hi = __builtin_convertvector(v, typename PK::bv);
                *(typename PK::bv*)&lds[0][4 * mq + c][kc] = hi;
                *(typename PK::bv*)&lds[1][4 * mq + c][kc] = __builtin_convertvector(
                    v - __builtin_convertvector(hi, typename PK::fv), typename PK::bv);
            }
        }
    }
}

// Column sums over k of a non-KFAST operand's staged slice (used for db):
// thread (mq, kg) adds its NQ k values of each of its four columns.
template <class Raw>
__device__ __forceinline__ void add_colsum(f4& cs, const Raw (&r)[NQ]) {
    f4 t = widen(r[0]);
#pragma unroll
    for (int j = 1; j < NQ; ++j) t += widen(r[j]);
    cs += t;
}

// Multiplies the staged 128 x BK slices: the wave's 4 x 4 blocks of 16 x 16,
// k-steps of 32.  Lane l supplies row l % 16 and k = 8 (l / 16) .. +7 of
// each fragment (the k order inside a step is irrelevant to the sum as long
// as A and B use the same one).
template <int PA, int PB>
__device__ __forceinline__ void mma_slice(__bf16 (*la)[BM][KP], __bf16 (*lb)[BN][KP],
                                          f4 (&acc)[4][4], int wm, int wn, int fr, int fk) {
#pragma unroll
    for (int ks = 0; ks < BK; ks += 32) {
        b8 fa[PA][4], fb[PB][4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
#pragma unroll
            for (int p = 0; p < PA; ++p)
                fa[p][i] = *(const b8*)&la[p][wm * 64 + i * 16 + fr][ks + fk];
#pragma unroll
            for (int p = 0; p < PB; ++p)
                fb[p][i] = *(const b8*)&lb[p][wn * 64 + i * 16 + fr][ks + fk];
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if constexpr (PB == 2)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[0][i], fb[1][j],
                                                                         acc[i][j], 0, 0, 0);
                if constexpr (PA == 2)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[1][i], fb[0][j],
                                                                         acc[i][j], 0, 0, 0);
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[0][i], fb[0][j],
                                                                     acc[i][j], 0, 0, 0);
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
// the four float4 values, and what epi.load fetched for those rows (strip 0's
// comes in as `pre`; strip i + 1's is fetched while strip i is stored).
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
        for (int q = 0; q < 4; ++q) val[q] = *(const f4*)&buf[(4 * q + (lane >> 4)) * EP + 4 * (lane & 15)];
        typename Epi::pre_t next{};
        if (i < 3) {
            int64_t mn[4];
            strip_rows(m0w, i + 1, lane, mn);
            epi.load(mn, n, next);
        }
        epi.run(m, n, val, pre);
        pre = next;
        __syncthreads();
    }
}

// A run of output tiles: tiles first, first + stride, ... (count of them),
// tile t at rows (t / ntn) * BM and columns (t % ntn) * BN, each the sum over
// k in [k_begin, k_end) of A(m, k) B(n, k), handed to epi.  The first
// K-slice of the next tile is fetched during the last slice of the current
// one, and so are the epilogue's reads of the destination.  If colsum_out is
// not null (A not KFAST, count 1), the sums over the same k range of the
// tile's 128 rows of A are written there.
template <class OpA, class OpB, class Epi>
__device__ __forceinline__ void tile_stream(const OpA& a, const OpB& b, int64_t k_begin,
                                            int64_t k_end, int64_t ntn, int64_t first,
                                            int64_t count, int64_t stride, const Epi& epi,
                                            char* smem, float* colsum_out = nullptr) {
    constexpr int PA = OpA::kPlanes, PB = OpB::kPlanes;
    __bf16 (*la)[BM][KP] = (__bf16 (*)[BM][KP])smem;
    __bf16 (*lb)[BN][KP] = (__bf16 (*)[BN][KP])(smem + (size_t)PA * BM * KP * 2);
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wv = tid >> 6;
    const int wm = wv >> 1, wn = wv & 1;
    const int fr = lane & 15, fk = 8 * (lane >> 4);
    const int64_t nsl = k_end > k_begin ? (k_end - k_begin + BK - 1) / BK : 0;
    if (count <= 0) return;

    typename OpA::raw_t ra[NQ];
    typename OpB::raw_t rb[NQ];
    f4 cs = f4{0.0f, 0.0f, 0.0f, 0.0f};
    int64_t t = first;
    if (nsl > 0) {
        fetch_slice(a, (t / ntn) * BM, k_begin, k_end, tid, ra);
        fetch_slice(b, (t % ntn) * BN, k_begin, k_end, tid, rb);
    }
    for (int64_t c = 0; c < count; ++c, t += stride) {
        const int64_t m0 = (t / ntn) * BM, n0 = (t % ntn) * BN;
        const int64_t m0w = m0 + wm * 64, n0w = n0 + wn * 64;
        f4 acc[4][4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = f4{0.0f, 0.0f, 0.0f, 0.0f};
        typename Epi::pre_t pre{};
        if (nsl == 0) {
            int64_t m[4];
            strip_rows(m0w, 0, lane, m);
            epi.load(m, n0w + 4 * (lane & 15), pre);
        }
        for (int64_t sl = 0; sl < nsl; ++sl) {
            store_slice<OpA>(la, tid, ra);
            store_slice<OpB>(lb, tid, rb);
            if constexpr (!OpA::kKFast)
                if (colsum_out) add_colsum(cs, ra);
            __syncthreads();
            if (sl + 1 < nsl) {
                const int64_t k0 = k_begin + (sl + 1) * BK;
                fetch_slice(a, m0, k0, k_end, tid, ra);
                fetch_slice(b, n0, k0, k_end, tid, rb);
            } else {
                if (c + 1 < count) {
                    const int64_t tn = t + stride;
                    fetch_slice(a, (tn / ntn) * BM, k_begin, k_end, tid, ra);
                    fetch_slice(b, (tn % ntn) * BN, k_begin, k_end, tid, rb);
                }
                int64_t m[4];
                strip_rows(m0w, 0, lane, m);
                epi.load(m, n0w + 4 * (lane & 15), pre);
            }
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
        tile_epilogue(acc, smem, m0w, n0w, epi, pre);
    }
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

template <typename T>
struct FwdEpi {
    struct pre_t {
        f4 bias;  // bias of the lane's four columns
    };
    float* zr;
    float* zi;
    const T* br;
    const T* bi;
    int64_t M, D;
    __device__ void load(const int64_t (&)[4], int64_t n, pre_t& pre) const {
        pre.bias = f4{0.0f, 0.0f, 0.0f, 0.0f};
        if (n >= 2 * D) return;
        const T* bp = n < D ? br : bi;
        const int64_t o = n < D ? n : n - D;
        if (bp) pre.bias = f4{recblr::load(bp + o), recblr::load(bp + o + 1), recblr::load(bp + o + 2), recblr::load(bp + o + 3)};
    }
    __device__ void run(const int64_t (&m)[4], int64_t n, const f4 (&v)[4],
                        const pre_t& pre) const {
        if (n >= 2 * D) return;
        float* base = n < D ? zr + n : zi + (n - D);
#pragma unroll
        for (int q = 0; q < 4; ++q)
            if (m[q] < M) *(f4*)(base + m[q] * D) = v[q] + pre.bias;
    }
};

// One 128 x 128 tile of [z_r | z_i] (M x 2D) per workgroup.
template <typename T>
__global__ __launch_bounds__(256, 2) void fwd_kernel(const T* x, const T* wr, const T* br,
                                                     const T* wi, const T* bi, float* zr,
                                                     float* zi, int64_t M, int64_t D) {
    using OpA = Operand<T, true, PlainMem<T>>;
    using OpB = Operand<T, true, RowPairMem<T>>;
    __shared__ __attribute__((aligned(16))) char smem[lds_bytes<OpA::kPlanes, OpB::kPlanes>()];
    const int64_t ntn = (2 * D + BN - 1) / BN;
    const int64_t t = xcd_tile(((M + BM - 1) / BM) * ntn);
    if (t < 0) return;
    const FwdEpi<T> epi{zr, zi, br, bi, M, D};
    tile_stream(OpA{{x, D}, M}, OpB{{wr, wi, D, D}, 2 * D}, 0, D, ntn, t, 1, 1, epi, smem);
}

template <typename T>
struct DxEpi {
    struct pre_t {
        f4 v[4];
    };
    T* dx;
    int64_t M, D;
    // dx holds the direct term delta * beta on entry.
    __device__ void load(const int64_t (&m)[4], int64_t n, pre_t& pre) const {
#pragma unroll
        for (int q = 0; q < 4; ++q)
            pre.v[q] = (n < D && m[q] < M) ? load_quad(dx + m[q] * D + n)
                                           : f4{0.0f, 0.0f, 0.0f, 0.0f};
    }
    __device__ void run(const int64_t (&m)[4], int64_t n, const f4 (&v)[4],
                        const pre_t& pre) const {
        if (n >= D) return;
        const f4(&old)[4] = pre.v;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if (m[q] >= M) continue;
            const f4 r = old[q] + v[q];
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

// One 128 x 128 tile of dx per workgroup.
template <typename T>
__global__ __launch_bounds__(256, 2) void dx_kernel(const float* dzr, const float* dzi,
                                                    const T* wr, const T* wi, T* dx, int64_t M,
                                                    int64_t D) {
    // A(m, k) = [dz_r | dz_i][m][k]; B(n, k) = Wcat[k][n], contiguous along n.
    using OpA = Operand<float, true, ColPairMem<float>>;
    using OpB = Operand<T, false, RowPairMem<T>>;
    __shared__ __attribute__((aligned(16))) char smem[lds_bytes<OpA::kPlanes, OpB::kPlanes>()];
    const int64_t ntn = (D + BN - 1) / BN;
    const int64_t t = xcd_tile(((M + BM - 1) / BM) * ntn);
    if (t < 0) return;
    const DxEpi<T> epi{dx, M, D};
    tile_stream(OpA{{dzr, dzi, D}, M}, OpB{{wr, wi, D, D}, D}, 0, 2 * D, ntn, t, 1, 1, epi,
                smem);
}

struct DwEpi {
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
// of [db_r; db_i]: dbpart[split][o].
template <typename T>
__global__ __launch_bounds__(256, 2) void dw_kernel(const float* dzr, const float* dzi,
                                                    const T* x,
                                                 float* partial, float* dbpart, int64_t M,
                                                 int64_t D, int64_t splits,
                                                 int64_t rows_per_split) {
    // A(o, row) = dz[row][o], B(k, row) = x[row][k]: both contiguous along o / k.
    using OpA = Operand<float, false, ColPairMem<float>>;
    using OpB = Operand<T, false, PlainMem<T>>;
    __shared__ __attribute__((aligned(16))) char smem[lds_bytes<OpA::kPlanes, OpB::kPlanes>()];
    __shared__ float colsum[BM];
    const int64_t nto = (2 * D + BM - 1) / BM, ntn = (D + BN - 1) / BN;
    const int64_t t = xcd_tile(nto * ntn * splits);
    if (t < 0) return;
    const int64_t split = t / (nto * ntn), tile = t % (nto * ntn);
    const int64_t to = tile / ntn, tn = tile % ntn;
    const int64_t k_begin = split * rows_per_split;
    const int64_t k_end = k_begin + rows_per_split < M ? k_begin + rows_per_split : M;
    const DwEpi epi{partial + split * (2 * D) * D, 2 * D, D};
    // The tiles of column block 0 also reduce db from the dz rows they stage.
    tile_stream(OpA{{dzr, dzi, D}, 2 * D}, OpB{{x, D}, D}, k_begin, k_end, ntn, tile, 1, 1, epi,
                smem, tn == 0 ? colsum : nullptr);
    if (tn == 0) {
        const int64_t o = to * BM + threadIdx.x;
        if (threadIdx.x < BM && o < 2 * D) dbpart[split * 2 * D + o] = colsum[threadIdx.x];
    }
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

int64_t dw_splits(int64_t M, int64_t D) {
    const int64_t tiles = ((2 * D + BM - 1) / BM) * ((D + BN - 1) / BN);
    int64_t splits = 512 / tiles;  // about two workgroups per CU
    const int64_t by_rows = (M + 511) / 512;  // at least 512 rows per split
    if (splits > by_rows) splits = by_rows;
    return splits < 1 ? 1 : splits;
}

}  // namespace fastmm

static bool fast_ok(int64_t D, std::initializer_list<const void*> ptrs) {
    if (D % 8 != 0) return false;
    for (const void* p : ptrs)
        if ((uintptr_t)p % 16 != 0) return false;
    return true;
}

// ------------------------------------------------------------------ launchers
static dim3 tiles(int64_t M, int64_t N, int64_t z = 1) {
    return dim3((unsigned)((M + kTM - 1) / kTM), (unsigned)((N + kTN - 1) / kTN), (unsigned)z);
}

hipError_t launch_project_forward(const void* x, const void* wr, const void* br, const void* wi,
                                  const void* bi, void* zr, void* zi, int64_t M, int64_t D,
                                  IoType io, hipStream_t stream) {
    if (M == 0 || D == 0) return hipSuccess;
    if (fast_ok(D, {x, wr, wi, zr, zi})) {
        const int64_t tiles = ((M + fastmm::BM - 1) / fastmm::BM) *
                              ((2 * D + fastmm::BN - 1) / fastmm::BN);
        if (io == IoType::kF32)
            hipLaunchKernelGGL(fastmm::fwd_kernel<float>, dim3(fastmm::grid_of(tiles)), dim3(256),
                               0, stream, (const float*)x, (const float*)wr, (const float*)br,
                               (const float*)wi, (const float*)bi, (float*)zr, (float*)zi, M, D);
        else
            hipLaunchKernelGGL(fastmm::fwd_kernel<bf16>, dim3(fastmm::grid_of(tiles)), dim3(256),
                               0, stream, (const bf16*)x, (const bf16*)wr, (const bf16*)br,
                               (const bf16*)wi, (const bf16*)bi, (float*)zr, (float*)zi, M, D);
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
                                        IoType io, hipStream_t stream) {
    if (M == 0 || D == 0) return hipSuccess;
    if (fast_ok(D, {dzr, dzi, wr, wi, dx})) {
        const int64_t tiles = ((M + fastmm::BM - 1) / fastmm::BM) *
                              ((D + fastmm::BN - 1) / fastmm::BN);
        if (io == IoType::kF32)
            hipLaunchKernelGGL(fastmm::dx_kernel<float>, dim3(fastmm::grid_of(tiles)), dim3(256),
                               0, stream, (const float*)dzr, (const float*)dzi, (const float*)wr,
                               (const float*)wi, (float*)dx, M, D);
        else
            hipLaunchKernelGGL(fastmm::dx_kernel<bf16>, dim3(fastmm::grid_of(tiles)), dim3(256),
                               0, stream, (const float*)dzr, (const float*)dzi, (const bf16*)wr,
                               (const bf16*)wi, (bf16*)dx, M, D);
        return hipGetLastError();
    }
    if (io == IoType::kF32)
        hipLaunchKernelGGL(proj_dx_kernel<float>, tiles(M, D), dim3(kThreads), 0, stream,
                           (const float*)dzr, (const float*)dzi, (const float*)wr,
                           (const float*)wi, (float*)dx, M, D);
    else
        hipLaunchKernelGGL(proj_dx_kernel<bf16>, tiles(M, D), dim3(kThreads), 0, stream,
                           (const float*)dzr, (const float*)dzi, (const bf16*)wr, (const bf16*)wi,
                           (bf16*)dx, M, D);
    return hipGetLastError();
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
    const size_t fast =
        (size_t)fastmm::dw_splits(M, D) * (size_t)(2 * D) * (size_t)(D + 1) * sizeof(float);
    return generic > fast ? generic : fast;
}

hipError_t launch_project_backward_weights(const void* dzr, const void* dzi, const void* x,
                                           float* dwr, float* dbr, float* dwi, float* dbi,
                                           int64_t M, int64_t D, IoType io, void* ws,
                                           hipStream_t stream) {
    if (D == 0) return hipSuccess;
    if (fast_ok(D, {dzr, dzi, x, ws})) {
        const int64_t splits = fastmm::dw_splits(M, D);
        const int64_t rows_per_split = (M + splits - 1) / splits;
        const int64_t tiles = ((2 * D + fastmm::BM - 1) / fastmm::BM) *
                              ((D + fastmm::BN - 1) / fastmm::BN) * splits;
        float* partial = (float*)ws;
        float* dbpart = partial + splits * 2 * D * D;
        if (io == IoType::kF32)
            hipLaunchKernelGGL(fastmm::dw_kernel<float>, dim3(fastmm::grid_of(tiles)), dim3(256),
                               0, stream, (const float*)dzr, (const float*)dzi, (const float*)x,
                               partial, dbpart, M, D, splits, rows_per_split);
        else
            hipLaunchKernelGGL(fastmm::dw_kernel<bf16>, dim3(fastmm::grid_of(tiles)), dim3(256),
                               0, stream, (const float*)dzr, (const float*)dzi, (const bf16*)x,
                               partial, dbpart, M, D, splits, rows_per_split);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        const int64_t total = 2 * D * D + 2 * D;
        hipLaunchKernelGGL(fastmm::dw_reduce_kernel, dim3((unsigned)((total + 63) / 64)),
                           dim3(64 * fastmm::kRedGroups), 0, stream, (const float*)partial, (const float*)dbpart,
                           splits, D, dwr, dbr, dwi, dbi);
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

}  // namespace recblr
