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

// The two trees of figure fig:scan over T2 leaves of nchw channels each
// (tr[p][k], composed in place): an up-sweep composes sibling ranges level by
// level (tree 1), a down-sweep hands every node the composition of all
// leaves before it (tree 2, root = identity).  On return tr[p] holds the
// exclusive prefix of leaf p.  All threads call it (it holds barriers).
__device__ __forceinline__ void two_tree_exclusive(float2* tr, int T2, int nchw, int tid) {
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
    two_tree_exclusive(tr, T2, nchw, tid);
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

// ------------------------------------------------------------------ backward
// The training side of the comparison: the same algorithms for the adjoint
// delta_t = dL/dh_t + alpha_{t+1} delta_{t+1} (delta_L = 0), which is the
// forward recurrence run backwards in time on the pairs
// (alpha_{t+1}, dL/dh_t), followed by the gate-gradient epilogue of the
// production backward.

// Gradients of one element from delta_t, the input x_t, the state h_{t-1}
// and the pre-activations (the production epilogue's arithmetic):
// dl is the element's term of dLambda before the sigmoid(Lambda) factor.
struct ElemGrad {
    float dx, dzr, dzi, dl;
};
__device__ __forceinline__ ElemGrad elem_grad(float delta, float hp, float x, float zr, float zi,
                                              const ChannelConst& cc) {
    const float r = sigmoid(zr), i = sigmoid(zi);
    const float al = fast_exp2(r * cc.neg_s_l2);
    const float q = r * cc.s;
    const float mm = one_minus_exp_neg(r * cc.two_s, al);
    const float rs = mm > 0.0f ? fast_rsq(mm) : 0.0f;
    const float sq = mm * rs;  // sqrt(1 - alpha^2)
    const float g_alpha = delta * hp, g_beta = delta * x;
    const float g1 = -al * g_alpha, g2 = g_beta * i * al * al;
    ElemGrad o;
    o.dl = fmaf(g1, r, g2 * (r * rs));
    o.dx = delta * sq * i;
    o.dzr = fmaf(g1, q, g2 * (q * rs)) * (1.0f - r);
    o.dzi = g_beta * sq * i * (1.0f - i);
    return o;
}

__device__ __forceinline__ float alpha_of(float zr, const ChannelConst& cc) {
    return fast_exp2(sigmoid(zr) * cc.neg_s_l2);
}

// Serial: one thread per channel walks the sequence from t = L - 1 down to 0
// (one wave per 64 channels, no parallelism along the sequence).
// partial[c]: the channel's dLambda term summed over t.
template <typename TX, typename TZ>
__global__ __launch_bounds__(kTreeThreads) void serial_bwd_kernel(
    const TX* x, const TZ* zr, const TZ* zi, const float* lam, const TX* h, const TX* dh, TX* dx,
    TZ* dzr, TZ* dzi, float* partial, int64_t L, int64_t D, int64_t nch) {
    const int64_t c = (int64_t)blockIdx.x * kTreeThreads + threadIdx.x;
    if (c >= nch) return;
    const int64_t b = c / D, d = c - b * D;
    const ChannelConst cc = channel_const(lam[d]);
    float delta = 0.0f, a_next = 0.0f, dsum = 0.0f;
    for (int64_t t = L - 1; t >= 0; --t) {
        const int64_t off = (b * L + t) * D + d;
        const float zrv = load(zr + off), ziv = load(zi + off);
        delta = fmaf(a_next, delta, load(dh + off));
        const float hp = t > 0 ? load(h + off - D) : 0.0f;
        const ElemGrad gr = elem_grad(delta, hp, load(x + off), zrv, ziv, cc);
        store(dx + off, gr.dx);
        store(dzr + off, gr.dzr);
        store(dzi + off, gr.dzi);
        dsum += gr.dl;
        a_next = alpha_of(zrv, cc);
    }
    partial[c] = dsum;
}

// Two-tree scan of the reversed sequence: leaf p holds step t = L - 1 - p
// (its pair (alpha_{t+1}, dL/dh_t)); leaves p >= L are the identity, the
// embedding padding of the forward seen from the other end.  Each thread
// keeps one channel (k = tid mod nchw) through the epilogue, so the dLambda
// terms are summed per thread in order and then over the threads of a
// channel in order.
template <typename TX, typename TZ>
__global__ __launch_bounds__(kTreeThreads) void tree_bwd_kernel(
    const TX* x, const TZ* zr, const TZ* zi, const float* lam, const TX* h, const TX* dh, TX* dx,
    TZ* dzr, TZ* dzi, float* partial, int64_t L, int64_t D, int64_t nch, int T2, int nchw) {
    extern __shared__ float2 sm[];
    float2* leaf = sm;
    float2* tr = sm + (size_t)T2 * nchw;
    __shared__ ChannelConst cct[64];
    __shared__ float red[kTreeThreads];
    const int tid = threadIdx.x;
    const int64_t c0 = (int64_t)blockIdx.x * nchw;
    if (tid < nchw && c0 + tid < nch) cct[tid] = channel_const(lam[(c0 + tid) % D]);
    __syncthreads();
    const int n = T2 * nchw;
    for (int e = tid; e < n; e += kTreeThreads) {
        const int p = e / nchw, k = e - p * nchw;
        const int64_t c = c0 + k, t = L - 1 - p;
        float2 v = make_float2(1.0f, 0.0f);
        if (c < nch && t >= 0) {
            const int64_t b = c / D, d = c - b * D;
            const int64_t off = (b * L + t) * D + d;
            const float a = t + 1 < L ? alpha_of(load(zr + off + D), cct[k]) : 0.0f;
            v = make_float2(a, load(dh + off));
        }
        leaf[e] = v;
        tr[e] = v;
    }
    __syncthreads();
    two_tree_exclusive(tr, T2, nchw, tid);
    float dsum = 0.0f;
    for (int e = tid; e < n; e += kTreeThreads) {
        const int p = e / nchw, k = e - p * nchw;
        const int64_t c = c0 + k, t = L - 1 - p;
        if (c < nch && t >= 0) {
            const int64_t b = c / D, d = c - b * D;
            const int64_t off = (b * L + t) * D + d;
            const float2 pre = tr[e], lf = leaf[e];
            const float delta = fmaf(lf.x, pre.y, lf.y);
            const float hp = t > 0 ? load(h + off - D) : 0.0f;
            const ElemGrad gr =
                elem_grad(delta, hp, load(x + off), load(zr + off), load(zi + off), cct[k]);
            store(dx + off, gr.dx);
            store(dzr + off, gr.dzr);
            store(dzi + off, gr.dzi);
            dsum += gr.dl;
        }
    }
    red[tid] = dsum;
    __syncthreads();
    if (tid < nchw && c0 + tid < nch) {
        float s = 0.0f;
        for (int j = tid; j < kTreeThreads; j += nchw) s += red[j];
        partial[c0 + tid] = s;
    }
}

// dLambda_d = sigmoid(Lambda_d) * sums[d].
__global__ __launch_bounds__(256) void dlambda_scale_kernel(const float* sums, const float* lam,
                                                            float* dlambda, int64_t D) {
    const int64_t d = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (d < D) dlambda[d] = sums[d] * sigmoid(lam[d]);
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

static size_t align256(size_t n) { return (n + 255) & ~(size_t)255; }

size_t scan_backward_method_workspace(int64_t B, int64_t D) {
    return align256((size_t)(B * D) * sizeof(float)) + align256((size_t)D * sizeof(float)) +
           colsum_workspace(B, D);
}

template <typename TX, typename TZ>
static hipError_t launch_bwd_method_t(bool tree, const ScanBwdArgs& a, float* partial,
                                      hipStream_t stream) {
    const int64_t nch = a.B * a.D;
    if (tree) {
        const int T2 = pow2_at_least(a.L);
        int nchw = (int)(kTreeLds / (2 * sizeof(float2) * (size_t)T2));
        if (nchw > 64) nchw = 64;
        if (nchw < 1) return hipErrorInvalidValue;
        const size_t lds = 2 * sizeof(float2) * (size_t)T2 * nchw;
        hipLaunchKernelGGL((tree_bwd_kernel<TX, TZ>), dim3((unsigned)((nch + nchw - 1) / nchw)),
                           dim3(kTreeThreads), lds, stream, (const TX*)a.x, (const TZ*)a.zr,
                           (const TZ*)a.zi, a.lambda, (const TX*)a.h, (const TX*)a.dh, (TX*)a.dx,
                           (TZ*)a.dzr, (TZ*)a.dzi, partial, a.L, a.D, nch, T2, nchw);
    } else {
        hipLaunchKernelGGL((serial_bwd_kernel<TX, TZ>),
                           dim3((unsigned)((nch + kTreeThreads - 1) / kTreeThreads)),
                           dim3(kTreeThreads), 0, stream, (const TX*)a.x, (const TZ*)a.zr,
                           (const TZ*)a.zi, a.lambda, (const TX*)a.h, (const TX*)a.dh, (TX*)a.dx,
                           (TZ*)a.dzr, (TZ*)a.dzi, partial, a.L, a.D, nch);
    }
    return hipGetLastError();
}

hipError_t launch_scan_backward_method(bool tree, const ScanBwdArgs& a, hipStream_t stream) {
    if (a.B * a.D == 0 || a.L == 0) return hipSuccess;
    char* ws = (char*)a.ws;
    float* partial = (float*)ws;
    float* sums = (float*)(ws + align256((size_t)(a.B * a.D) * sizeof(float)));
    void* cws = ws + align256((size_t)(a.B * a.D) * sizeof(float)) +
                align256((size_t)a.D * sizeof(float));
    const hipError_t e = a.io == IoType::kF32
                             ? launch_bwd_method_t<float, float>(tree, a, partial, stream)
                             : launch_bwd_method_t<bf16, bf16>(tree, a, partial, stream);
    if (e != hipSuccess) return e;
    // dLambda: the per-channel sums over b in a fixed order, then sigmoid(Lambda).
    const hipError_t e2 = launch_colsum(partial, a.B, a.D, sums, cws, stream);
    if (e2 != hipSuccess) return e2;
    hipLaunchKernelGGL(dlambda_scale_kernel, dim3((unsigned)((a.D + 255) / 256)), dim3(256), 0,
                       stream, sums, a.lambda, a.dlambda, a.D);
    return hipGetLastError();
}

}  // namespace recblr
