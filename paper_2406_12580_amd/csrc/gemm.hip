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

// ------------------------------------------------------------------ launchers
static dim3 tiles(int64_t M, int64_t N, int64_t z = 1) {
    return dim3((unsigned)((M + kTM - 1) / kTM), (unsigned)((N + kTN - 1) / kTN), (unsigned)z);
}

hipError_t launch_project_forward(const void* x, const void* wr, const void* br, const void* wi,
                                  const void* bi, void* zr, void* zi, int64_t M, int64_t D,
                                  IoType io, hipStream_t stream) {
    if (M == 0 || D == 0) return hipSuccess;
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
    return (size_t)project_dw_splits(M, D) * (size_t)(2 * D) * (size_t)(D + 1) * sizeof(float);
}

hipError_t launch_project_backward_weights(const void* dzr, const void* dzi, const void* x,
                                           float* dwr, float* dbr, float* dwi, float* dbi,
                                           int64_t M, int64_t D, IoType io, void* ws,
                                           hipStream_t stream) {
    if (D == 0) return hipSuccess;
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
