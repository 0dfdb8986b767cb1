// Parallel-scan variants for the efficiency ablation of RecBLR (arXiv
// 2406.12580, section 4, Table tab:efficiency): the paper's two-tree scan
// (section 3.3, figure fig:scan) over a power-of-two length, with the
// embedding padding of section 3.3 applied inside the kernel.  The
// production kernels (scan_fwd.hip) need no padding; this one exists to
// measure the algorithms against each other on the same inputs.
//
// One workgroup holds nchw channels x T2 steps of (alpha, beta') pairs in LDS
// (T2 = the power of two >= L).  The first T2 - L positions are the identity
// (1, 0): with a zero initial state this is exactly left padding with zero
// embeddings.  An up-sweep composes pairs level by level (tree 1), a
// down-sweep hands every node the composition of everything before it
// (tree 2, root = identity), and h_t = c_t . prefix_t.
#include "device_common.hpp"
#include "launch.hpp"

namespace recblr {

namespace {
constexpr int kTreeThreads = 256;
constexpr int kTreeMaxSteps = 4096;
constexpr size_t kTreeLds = 64 * 1024;  // two arrays of T2 * nchw float2

__device__ __forceinline__ float2 later_after(float2 later, float2 earlier) {
    return make_float2(later.x * earlier.x, fmaf(later.x, earlier.y, later.y));
}
}  // namespace

template <typename TX, typename TZ>
__global__ __launch_bounds__(kTreeThreads) void tree_fwd_kernel(const TX* x, const TZ* zr,
                                                                const TZ* zi, const float* lam,
                                                                TX* h, int64_t L, int64_t D,
                                                                int64_t nch, int T2, int nchw) {
    extern __shared__ float2 sm[];
    float2* leaf = sm;                      // [T2][nchw] pairs c_t
    float2* tr = sm + (size_t)T2 * nchw;    // [T2][nchw] tree nodes (in place)
    __shared__ ChannelConst cct[64];
    const int tid = threadIdx.x;
    const int64_t c0 = (int64_t)blockIdx.x * nchw;
    const int pad = T2 - (int)L;
    if (tid < nchw && c0 + tid < nch) cct[tid] = channel_const(lam[(c0 + tid) % D]);
    __syncthreads();
    const int n = T2 * nchw;
    for (int e = tid; e < n; e += kTreeThreads) {
        const int p = e / nchw, k = e - p * nchw;
        const int64_t c = c0 + k, t = (int64_t)p - pad;
        float2 v = make_float2(1.0f, 0.0f);
        if (c < nch && t >= 0) {
            const int64_t b = c / D, d = c - b * D;
            const int64_t off = (b * L + t) * D + d;
            float a, u;
            gate_forward(load(x + off), load(zr + off), load(zi + off), cct[k], a, u);
            v = make_float2(a, u);
        }
        leaf[e] = v;
        tr[e] = v;
    }
    __syncthreads();
    // Up-sweep: node hi of each pair of sibling ranges takes later . earlier.
    for (int s = 1; s < T2; s <<= 1) {
        const int nodes = T2 / (2 * s) * nchw;
        for (int e = tid; e < nodes; e += kTreeThreads) {
            const int j = e / nchw, k = e - j * nchw;
            const int hi = 2 * s * j + 2 * s - 1, lo = hi - s;
            tr[hi * nchw + k] = later_after(tr[hi * nchw + k], tr[lo * nchw + k]);
        }
        __syncthreads();
    }
    // Down-sweep: the earlier half inherits the node's prefix, the later half
    // gets (total of the earlier half) . prefix.
    if (tid < nchw) tr[(T2 - 1) * nchw + tid] = make_float2(1.0f, 0.0f);
    __syncthreads();
    for (int s = T2 / 2; s >= 1; s >>= 1) {
        const int nodes = T2 / (2 * s) * nchw;
        for (int e = tid; e < nodes; e += kTreeThreads) {
            const int j = e / nchw, k = e - j * nchw;
            const int hi = 2 * s * j + 2 * s - 1, mid = hi - s;
            const float2 pre = tr[hi * nchw + k], tot_e = tr[mid * nchw + k];
            tr[mid * nchw + k] = pre;
            tr[hi * nchw + k] = later_after(tot_e, pre);
        }
        __syncthreads();
    }
    for (int e = tid; e < n; e += kTreeThreads) {
        const int p = e / nchw, k = e - p * nchw;
        const int64_t c = c0 + k, t = (int64_t)p - pad;
        if (c < nch && t >= 0) {
            const int64_t b = c / D, d = c - b * D;
            const float2 pre = tr[e], lf = leaf[e];
            store(h + (b * L + t) * D + d, fmaf(lf.x, pre.y, lf.y));
        }
    }
}

static int pow2_at_least(int64_t L) {
    int t = 1;
    while (t < L) t <<= 1;
    return t;
}

bool tree_scan_supported(int64_t L) { return L <= kTreeMaxSteps; }

hipError_t launch_scan_forward_tree(const ScanFwdArgs& a, hipStream_t stream) {
    const int64_t nch = a.B * a.D;
    if (nch == 0 || a.L == 0) return hipSuccess;
    const int T2 = pow2_at_least(a.L);
    int nchw = (int)(kTreeLds / (2 * sizeof(float2) * (size_t)T2));
    if (nchw > 64) nchw = 64;
    if (nchw < 1) return hipErrorInvalidValue;
    const size_t lds = 2 * sizeof(float2) * (size_t)T2 * nchw;
    const dim3 grid((unsigned)((nch + nchw - 1) / nchw));
    if (a.io == IoType::kF32)
        hipLaunchKernelGGL((tree_fwd_kernel<float, float>), grid, dim3(kTreeThreads), lds, stream,
                           (const float*)a.x, (const float*)a.zr, (const float*)a.zi, a.lambda,
                           (float*)a.h, a.L, a.D, nch, T2, nchw);
    else
        hipLaunchKernelGGL((tree_fwd_kernel<bf16, bf16>), grid, dim3(kTreeThreads), lds, stream,
                           (const bf16*)a.x, (const bf16*)a.zr, (const bf16*)a.zi, a.lambda,
                           (bf16*)a.h, a.L, a.D, nch, T2, nchw);
    return hipGetLastError();
}

}  // namespace recblr
