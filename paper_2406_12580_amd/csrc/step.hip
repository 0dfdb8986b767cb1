// One recurrent step of the BD-LRU for inference (RecBLR, arXiv 2406.12580,
// eq:linrnn with the gates of section 3.2):
//   h_next[b, d] = alpha(z_r) h_prev[b, d] + beta(z_r, z_i) x[b, d]
// Purely elementwise and bound by HBM bandwidth.  Each thread handles 8
// consecutive elements (one 16-byte bf16 load or two 16-byte fp32 loads per
// operand); the per-channel constants of softplus(Lambda) are built once per
// workgroup in LDS and the grid strides over the [B, D] array.
#include "device_common.hpp"
#include "launch.hpp"

namespace recblr {

constexpr int kStepThreads = 256;
constexpr int kStepVec = 8;
constexpr int kStepMaxTable = 2048;  // channels whose constants fit the LDS table

template <typename T>
struct Vec8;

template <>
struct Vec8<float> {
    float4 lo, hi;
    __device__ __forceinline__ void load(const float* p) {
        lo = *(const float4*)p;
        hi = *(const float4*)(p + 4);
    }
    __device__ __forceinline__ float get(int k) const {
        const float* f = k < 4 ? &lo.x : &hi.x;
        return f[k & 3];
    }
};

template <>
struct Vec8<bf16> {
    uint4 raw;
    __device__ __forceinline__ void load(const bf16* p) { raw = *(const uint4*)p; }
    __device__ __forceinline__ float get(int k) const {
        const uint32_t* w = &raw.x;
        uint32_t word = w[k >> 1];
        return __uint_as_float((k & 1) ? (word & 0xFFFF0000u) : (word << 16));
    }
};

// Vector path: n and D multiples of 8, every pointer 16-byte aligned, D <= table size.
template <typename T, typename TZ>
__global__ __launch_bounds__(kStepThreads) void step_vec_kernel(
    const T* __restrict__ x, const TZ* __restrict__ zr, const TZ* __restrict__ zi,
    const float* __restrict__ lam, const float* h_prev, float* h_next, int64_t n, int64_t D) {
    __shared__ ChannelConst table[kStepMaxTable];
    for (int64_t d = threadIdx.x; d < D; d += blockDim.x) table[d] = channel_const(lam[d]);
    __syncthreads();
    const int64_t stride = (int64_t)gridDim.x * blockDim.x * kStepVec;
    for (int64_t e0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * kStepVec; e0 < n;
         e0 += stride) {
        Vec8<T> vx;
        Vec8<TZ> vr, vi;
        vx.load(x + e0);
        vr.load(zr + e0);
        vi.load(zi + e0);
        float4 hp0 = *(const float4*)(h_prev + e0);
        float4 hp1 = *(const float4*)(h_prev + e0 + 4);
        float hp[8] = {hp0.x, hp0.y, hp0.z, hp0.w, hp1.x, hp1.y, hp1.z, hp1.w};
        float out[8];
        const int64_t d0 = e0 % D;
#pragma unroll
        for (int k = 0; k < kStepVec; ++k) {
            float a, u;
            gate_forward(vx.get(k), vr.get(k), vi.get(k), table[d0 + k], a, u);
            out[k] = fmaf(a, hp[k], u);
        }
        *(float4*)(h_next + e0) = make_float4(out[0], out[1], out[2], out[3]);
        *(float4*)(h_next + e0 + 4) = make_float4(out[4], out[5], out[6], out[7]);
    }
}

// General path: any alignment and any D.
template <typename T, typename TZ>
__global__ __launch_bounds__(kStepThreads) void step_scalar_kernel(
    const T* __restrict__ x, const TZ* __restrict__ zr, const TZ* __restrict__ zi,
    const float* __restrict__ lam, const float* h_prev, float* h_next, int64_t n, int64_t D) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += stride) {
        float a, u;
        gate_forward(load(x + e), load(zr + e), load(zi + e), channel_const(lam[e % D]), a, u);
        h_next[e] = fmaf(a, h_prev[e], u);
    }
}

static bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

template <typename T, typename TZ>
static hipError_t launch_step_t(const void* x, const void* zr, const void* zi, const float* lam,
                                const float* h_prev, float* h_next, int64_t B, int64_t D,
                                hipStream_t stream) {
    const int64_t n = B * D;
    if (n == 0) return hipSuccess;
    const bool vec = (D % kStepVec == 0) && D <= kStepMaxTable && aligned16(x) &&
                     aligned16(zr) && aligned16(zi) && aligned16(h_prev) && aligned16(h_next);
    if (vec) {
        int64_t blocks = (n / kStepVec + kStepThreads - 1) / kStepThreads;
        if (blocks > 2048) blocks = 2048;
        hipLaunchKernelGGL((step_vec_kernel<T, TZ>), dim3((unsigned)blocks), dim3(kStepThreads),
                           0, stream, (const T*)x, (const TZ*)zr, (const TZ*)zi, lam, h_prev,
                           h_next, n, D);
    } else {
        int64_t blocks = (n + kStepThreads - 1) / kStepThreads;
        if (blocks > 8192) blocks = 8192;
        hipLaunchKernelGGL((step_scalar_kernel<T, TZ>), dim3((unsigned)blocks),
                           dim3(kStepThreads), 0, stream, (const T*)x, (const TZ*)zr,
                           (const TZ*)zi, lam, h_prev, h_next, n, D);
    }
    return hipGetLastError();
}

hipError_t launch_scan_step(const void* x, const void* zr, const void* zi, const float* lambda,
                            const float* h_prev, float* h_next, int64_t B, int64_t D, IoType io,
                            IoType zio, hipStream_t stream) {
    if (io == IoType::kF32)
        return launch_step_t<float, float>(x, zr, zi, lambda, h_prev, h_next, B, D, stream);
    if (zio == IoType::kF32)
        return launch_step_t<bf16, float>(x, zr, zi, lambda, h_prev, h_next, B, D, stream);
    return launch_step_t<bf16, bf16>(x, zr, zi, lambda, h_prev, h_next, B, D, stream);
}

}  // namespace recblr
