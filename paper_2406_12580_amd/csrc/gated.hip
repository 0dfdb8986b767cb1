// Gated recurrent layer core of RecBLR (arXiv 2406.12580, Algorithm
// alg:gated_recurrent, lines 3 to 5) outside the fused scan: the causal
// depthwise Conv1d + SiLU that forms the BD-LRU input, and the output gate
// y = h * SiLU(hz).  The scan kernel with the projections fused in applies
// both on the fly; these kernels serve the shapes it does not cover.
#include "device_common.hpp"
#include "launch.hpp"

namespace recblr {

namespace {
constexpr int kGateThreads = 256;
}

// Taps as [kConvTaps][D] (zero past K) and the bias as [D] (zero if none).
__global__ void pack_conv_kernel(const float* __restrict__ w, const float* __restrict__ b, int K,
                                 int64_t D, float* __restrict__ w4, float* __restrict__ b4) {
    const int64_t d = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (d >= D) return;
#pragma unroll
    for (int j = 0; j < kConvTaps; ++j) w4[j * D + d] = j < K ? w[d * K + j] : 0.0f;
    b4[d] = b ? b[d] : 0.0f;
}

// x'_t = SiLU(b + sum_j w_j hx_{t-j}) with hx_{t<0} = 0, one element per thread.
template <typename T>
__global__ __launch_bounds__(kGateThreads) void conv_silu_kernel(const T* __restrict__ hx,
                                                                 const float* __restrict__ w4,
                                                                 const float* __restrict__ b4,
                                                                 T* __restrict__ xp, int64_t L,
                                                                 int64_t D, int64_t n) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= n) return;
    const int64_t d = e % D, t = (e / D) % L;
    float c = b4[d];
#pragma unroll
    for (int j = 0; j < kConvTaps; ++j)
        if (t - j >= 0) c = fmaf(w4[j * D + d], load(hx + e - j * D), c);
    store(xp + e, c * sigmoid(c));
}

// The same with 16-byte accesses: V = 16 / sizeof(T) consecutive channels per
// thread (D % V == 0, 16-byte aligned tensors).
template <typename T>
__global__ __launch_bounds__(kGateThreads) void conv_silu_vec_kernel(
    const T* __restrict__ hx, const float* __restrict__ w4, const float* __restrict__ b4,
    T* __restrict__ xp, int64_t L, int64_t D, int64_t nvec) {
    constexpr int V = 16 / sizeof(T);
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= nvec) return;
    const int64_t e = q * V;
    const int64_t d = e % D, t = (e / D) % L;
    float c[V];
#pragma unroll
    for (int i = 0; i < V; ++i) c[i] = b4[d + i];
#pragma unroll
    for (int j = 0; j < kConvTaps; ++j) {
        if (t - j < 0) break;
        const uint4 raw = *(const uint4*)(hx + e - j * D);
        const T* v = (const T*)&raw;
#pragma unroll
        for (int i = 0; i < V; ++i) c[i] = fmaf(w4[j * D + d + i], to_f32(v[i]), c[i]);
    }
    uint4 out;
    T* o = (T*)&out;
#pragma unroll
    for (int i = 0; i < V; ++i) o[i] = from_f32<T>(c[i] * sigmoid(c[i]));
    *(uint4*)(xp + e) = out;
}

template <typename T>
__global__ __launch_bounds__(kGateThreads) void gate_out_kernel(const T* __restrict__ h,
                                                                const T* __restrict__ hz,
                                                                T* __restrict__ y, int64_t n) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= n) return;
    const float g = load(hz + e);
    store(y + e, load(h + e) * (g * sigmoid(g)));
}

template <typename T>
__global__ __launch_bounds__(kGateThreads) void gate_out_vec_kernel(const T* __restrict__ h,
                                                                    const T* __restrict__ hz,
                                                                    T* __restrict__ y,
                                                                    int64_t nvec) {
    constexpr int V = 16 / sizeof(T);
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= nvec) return;
    const uint4 rh = *(const uint4*)(h + q * V), rz = *(const uint4*)(hz + q * V);
    const T* vh = (const T*)&rh;
    const T* vz = (const T*)&rz;
    uint4 out;
    T* o = (T*)&out;
#pragma unroll
    for (int i = 0; i < V; ++i) {
        const float g = to_f32(vz[i]);
        o[i] = from_f32<T>(to_f32(vh[i]) * (g * sigmoid(g)));
    }
    *(uint4*)(y + q * V) = out;
}

hipError_t launch_pack_conv(const float* w, const float* b, int K, int64_t D, float* w4,
                            float* b4, hipStream_t stream) {
    hipLaunchKernelGGL(pack_conv_kernel, dim3((unsigned)((D + 255) / 256)), dim3(256), 0, stream,
                       w, b, K, D, w4, b4);
    return hipGetLastError();
}

hipError_t launch_conv_silu(const void* hx, const float* w4, const float* b4, void* xp, int64_t B,
                            int64_t L, int64_t D, IoType io, hipStream_t stream) {
    const int64_t n = B * L * D;
    if (n == 0) return hipSuccess;
    const int V = io == IoType::kF32 ? 4 : 8;
    if (D % V == 0 && ((uintptr_t)hx | (uintptr_t)xp) % 16 == 0) {
        const int64_t nvec = n / V;
        const dim3 grid((unsigned)((nvec + kGateThreads - 1) / kGateThreads));
        if (io == IoType::kF32)
            hipLaunchKernelGGL(conv_silu_vec_kernel<float>, grid, dim3(kGateThreads), 0, stream,
                               (const float*)hx, w4, b4, (float*)xp, L, D, nvec);
        else
            hipLaunchKernelGGL(conv_silu_vec_kernel<bf16>, grid, dim3(kGateThreads), 0, stream,
                               (const bf16*)hx, w4, b4, (bf16*)xp, L, D, nvec);
        return hipGetLastError();
    }
    const dim3 grid((unsigned)((n + kGateThreads - 1) / kGateThreads));
    if (io == IoType::kF32)
        hipLaunchKernelGGL(conv_silu_kernel<float>, grid, dim3(kGateThreads), 0, stream,
                           (const float*)hx, w4, b4, (float*)xp, L, D, n);
    else
        hipLaunchKernelGGL(conv_silu_kernel<bf16>, grid, dim3(kGateThreads), 0, stream,
                           (const bf16*)hx, w4, b4, (bf16*)xp, L, D, n);
    return hipGetLastError();
}

hipError_t launch_gate_out(const void* h, const void* hz, void* y, int64_t n, IoType io,
                           hipStream_t stream) {
    if (n == 0) return hipSuccess;
    const int V = io == IoType::kF32 ? 4 : 8;
    if (n % V == 0 && ((uintptr_t)h | (uintptr_t)hz | (uintptr_t)y) % 16 == 0) {
        const int64_t nvec = n / V;
        const dim3 grid((unsigned)((nvec + kGateThreads - 1) / kGateThreads));
        if (io == IoType::kF32)
            hipLaunchKernelGGL(gate_out_vec_kernel<float>, grid, dim3(kGateThreads), 0, stream,
                               (const float*)h, (const float*)hz, (float*)y, nvec);
        else
            hipLaunchKernelGGL(gate_out_vec_kernel<bf16>, grid, dim3(kGateThreads), 0, stream,
                               (const bf16*)h, (const bf16*)hz, (bf16*)y, nvec);
        return hipGetLastError();
    }
    const dim3 grid((unsigned)((n + kGateThreads - 1) / kGateThreads));
    if (io == IoType::kF32)
        hipLaunchKernelGGL(gate_out_kernel<float>, grid, dim3(kGateThreads), 0, stream,
                           (const float*)h, (const float*)hz, (float*)y, n);
    else
        hipLaunchKernelGGL(gate_out_kernel<bf16>, grid, dim3(kGateThreads), 0, stream,
                           (const bf16*)h, (const bf16*)hz, (bf16*)y, n);
    return hipGetLastError();
}

}  // namespace recblr
