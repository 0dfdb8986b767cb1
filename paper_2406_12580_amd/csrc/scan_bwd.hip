// Backward BD-LRU scan for gfx950: a reverse-direction chunked scan of the
// adjoint with the gate-gradient epilogue fused into it, then a deterministic
// reduction of dLoss/dLambda.
//
// The forward recurrence is h_t = alpha_t h_{t-1} + beta_t x_t (RecBLR,
// arXiv 2406.12580, eq:linrnn) with the gates of section 3.2.  Its adjoint,
// with G_t = dLoss/dh_t, is the same first-order recurrence run backwards:
//   delta_t = G_t + alpha_{t+1} delta_{t+1},   delta_{L+1} = 0  (+ dhT at t = L)
// so it reuses the forward machinery with the pair (alpha_{t+1}, G_t) per step
// and carries flowing from later to earlier steps.  Per element, with
// q = softplus(Lambda) r, m = 1 - alpha^2 and rs = 1/sqrt(m):
//   g_alpha = delta_t h_{t-1},  g_beta = delta_t x_t,  dx = delta_t beta_t
//   dLoss/dq = -alpha g_alpha + g_beta i alpha^2 rs
//   dz_r = dLoss/dq * q (1 - r),   dz_i = g_beta sqrt(m) i (1 - i)
//   dLoss/dLambda = sigmoid(Lambda) * sum_{b,t} dLoss/dq * r
//   dh0 = alpha_1 delta_1
// The paper gives no backward pass; these are the exact derivatives of its
// forward equations.
//
// Decomposition mirrors the forward chain kernel: lane = channel, workgroup =
// 64 channels x the whole sequence, W waves per macro-chunk of W*C steps,
// macro-chunks visited from the end of the sequence to its start.
#include "device_common.hpp"
#include "launch.hpp"

namespace recblr {

namespace {

constexpr size_t kAlign = 256;
inline size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// Rows of the per-channel dLambda partials are reduced in blocks of this many.
constexpr int kReduceRows = 64;

struct BwdWorkspace {
    unsigned* counter;  // arrival counter of the reduction's last-block step
    float* partial;     // [rows][D] per-channel sums of dLoss/dq * r
    double* partial2;   // [ceil(rows / kReduceRows)][D]
};

inline size_t bwd_ws_bytes(int64_t rows, int64_t D) {
    int64_t nb = (rows + kReduceRows - 1) / kReduceRows;
    return kAlign + align_up((size_t)(rows * D) * sizeof(float)) +
           align_up((size_t)(nb * D) * sizeof(double));
}

inline BwdWorkspace bwd_ws_carve(void* ws, int64_t rows, int64_t D) {
    char* p = (char*)ws;
    BwdWorkspace w;
    w.counter = (unsigned*)p;
    p += kAlign;
    w.partial = (float*)p;
    p += align_up((size_t)(rows * D) * sizeof(float));
    w.partial2 = (double*)p;
    return w;
}

}  // namespace

template <typename T, typename TZ, int C, typename Off>
struct BwdRegs {
    float g[C], x[C], zr[C], zi[C], hp[C];
    float zr_after;  // z_r of the step just after this wave's chunk

    // Loads steps [t_first, t_first + C) (clamped to L-1; the caller masks) and
    // h_{t-1} for each of them (h0 at t = 0).
    __device__ __forceinline__ void fetch(const T* __restrict__ G, const T* __restrict__ X,
                                          const TZ* __restrict__ ZR, const TZ* __restrict__ ZI,
                                          const T* __restrict__ H, float h0v, Off base, Off row,
                                          int64_t t_first, int64_t L) {
#pragma unroll
        for (int j = 0; j < C; ++j) {
            int64_t t = t_first + j < L ? t_first + j : L - 1;
            Off off = base + (Off)t * row;
            g[j] = load_at(G, off);
            x[j] = load_at(X, off);
            zr[j] = load_at(ZR, z_offset<T, TZ>(off));
            zi[j] = load_at(ZI, z_offset<T, TZ>(off));
            float hv = load_at(H, t > 0 ? off - row : off);
            hp[j] = t > 0 ? hv : h0v;
        }
        int64_t ta = t_first + C < L ? t_first + C : L - 1;
        zr_after = load_at(ZR, z_offset<T, TZ>(base + (Off)ta * row));
    }
};

template <typename T, typename TZ, int W, int C, typename Off>
__global__ __launch_bounds__(W* kWave) void scan_bwd_chain_kernel(
    const T* __restrict__ X, const TZ* __restrict__ ZR, const TZ* __restrict__ ZI,
    const float* __restrict__ lam, const float* __restrict__ h0, const T* __restrict__ H,
    const T* __restrict__ G, const float* __restrict__ dhT, T* __restrict__ DX,
    TZ* __restrict__ DZR, TZ* __restrict__ DZI, float* __restrict__ dh0,
    float* __restrict__ partial, unsigned* __restrict__ counter, int64_t L, int64_t D,
    int64_t nch) {
    __shared__ Seg agg[2][W][kWave];
    __shared__ float red[W][kWave];
    if (blockIdx.x == 0 && threadIdx.x == 0) *counter = 0u;  // consumed by the reduction

    const int lane = threadIdx.x & (kWave - 1);
    const int w = threadIdx.x / kWave;
    const int64_t c = (int64_t)blockIdx.x * kWave + lane;
    const bool valid = c < nch;
    const int64_t cs = valid ? c : 0;  // idle lanes shadow channel 0 and store nothing
    const int64_t b = cs / D;
    const int64_t d = cs - b * D;
    const Off base = (Off)((b * L * D + d) * (int64_t)sizeof(T));
    const Off row = (Off)(D * (int64_t)sizeof(T));
    const ChannelConst cc = channel_const(lam[d]);
    const float h0v = h0 ? h0[cs] : 0.0f;
    const float dhTv = dhT ? dhT[cs] : 0.0f;

    constexpr int64_t kMacro = (int64_t)W * C;
    const int64_t nmacro = (L + kMacro - 1) / kMacro;
    float carry = 0.0f;   // delta flowing in from later steps
    float dsum = 0.0f;    // sum of dLoss/dq * r over this lane's steps

    BwdRegs<T, TZ, C, Off> cur, nxt;
    if (nmacro > 0)
        cur.fetch(G, X, ZR, ZI, H, h0v, base, row, (nmacro - 1) * kMacro + (int64_t)w * C, L);
    int buf = 0;
    for (int64_t m = nmacro - 1; m >= 0; --m, buf ^= 1) {
        const int64_t tw = m * kMacro + (int64_t)w * C;
        if (m > 0) nxt.fetch(G, X, ZR, ZI, H, h0v, base, row, tw - kMacro, L);

        // alpha_t and r_t of this chunk; alpha of the step after it.
        float r[C], al[C], ap[C], gg[C];
#pragma unroll
        for (int j = 0; j < C; ++j) {
            r[j] = sigmoid(cur.zr[j]);
            al[j] = fast_exp2(r[j] * cc.neg_s_l2);
        }
        const float al_after = fast_exp2(sigmoid(cur.zr_after) * cc.neg_s_l2);
#pragma unroll
        for (int j = 0; j < C; ++j) {
            const int64_t t = tw + j;
            const bool ok = t < L;
            float nxt_alpha = (j + 1 < C) ? al[j + 1 < C ? j + 1 : j] : al_after;
            if (t + 1 >= L) nxt_alpha = 0.0f;    // delta_{L+1} = 0
            const float gj = cur.g[j] + (t == L - 1 ? dhTv : 0.0f);
            ap[j] = ok ? nxt_alpha : 1.0f;       // steps past the end are the identity (1, 0)
            gg[j] = ok ? gj : 0.0f;
        }
        // Local aggregate of the reverse recurrence over this wave's chunk.
        Seg s{1.0f, 0.0f};
#pragma unroll
        for (int j = C - 1; j >= 0; --j) s = compose(Seg{ap[j], gg[j]}, s);
        agg[buf][w][lane] = s;
        __syncthreads();

        // Carry into this wave: fold the later waves, last one first.
        float cin = carry;
#pragma unroll
        for (int k = W - 1; k >= 0; --k) {
            if (k > w) {
                Seg e = agg[buf][k][lane];
                cin = fmaf(e.A, cin, e.H);
            }
        }
        // Re-run the chunk backwards from the true carry; gate-gradient epilogue.
        float delta = cin;
#pragma unroll
        for (int j = C - 1; j >= 0; --j) {
            delta = fmaf(ap[j], delta, gg[j]);
            const int64_t t = tw + j;
            if (t < L) {
                const float i = sigmoid(cur.zi[j]);
                const float q = r[j] * cc.s;
                const float mm = one_minus_exp_neg(r[j] * cc.two_s, al[j]);
                const float rs = mm > 0.0f ? fast_rsq(mm) : 0.0f;
                const float sq = mm * rs;  // sqrt(1 - alpha^2)
                const float g_alpha = delta * cur.hp[j];
                const float g_beta = delta * cur.x[j];
                const float g1 = -al[j] * g_alpha;
                const float g2 = g_beta * i * al[j] * al[j];
                dsum = fmaf(g1, r[j], fmaf(g2, r[j] * rs, dsum));
                if (valid) {
                    const Off off = base + (Off)t * row;
                    store_at(DX, off, delta * sq * i);
                    const Off zoff = z_offset<T, TZ>(off);
                    store_at(DZR, zoff, fmaf(g1, q, g2 * (q * rs)) * (1.0f - r[j]));
                    store_at(DZI, zoff, g_beta * sq * i * (1.0f - i));
                    if (t == 0 && dh0) dh0[cs] = al[j] * delta;
                }
            }
        }
        // Carry out of the macro-chunk (towards earlier steps).
        float cout = cin;
#pragma unroll
        for (int k = W - 1; k >= 0; --k) {
            if (k <= w) {
                Seg e = agg[buf][k][lane];
                cout = fmaf(e.A, cout, e.H);
            }
        }
        carry = cout;
        cur = nxt;
    }
    if (L == 0 && w == 0 && valid && dh0) dh0[cs] = dhTv;

    // Per-channel partial of dLoss/dLambda: waves combined in a fixed order.
    red[w][lane] = dsum;
    __syncthreads();
    if (w == 0 && valid) {
        float acc = 0.0f;
#pragma unroll
        for (int k = 0; k < W; ++k) acc += red[k][lane];
        partial[cs] = acc;
    }
}

// dLambda[d] = sigmoid(Lambda_d) * sum_rows partial[row][d], in double, in a
// fixed order.  Block (nb, dg) sums rows [nb*64, nb*64 + 64) of channels
// [dg*64, dg*64 + 64); the last block to arrive adds the block sums in
// row-block order.
__global__ __launch_bounds__(256) void dlambda_reduce_kernel(
    const float* __restrict__ partial, double* __restrict__ partial2, unsigned* counter,
    const float* __restrict__ lam, float* __restrict__ dlambda, int64_t rows, int64_t D) {
    __shared__ double red[4][kWave];
    __shared__ bool last;
    const int lane = threadIdx.x & (kWave - 1);
    const int w = threadIdx.x / kWave;
    const int64_t d = (int64_t)blockIdx.y * kWave + lane;
    const int64_t nb = blockIdx.x;
    double acc = 0.0;
    if (d < D) {
        int64_t r0 = nb * kReduceRows + w * (kReduceRows / 4);
#pragma unroll
        for (int k = 0; k < kReduceRows / 4; ++k) {
            int64_t row = r0 + k;
            if (row < rows) acc += (double)partial[row * D + d];
        }
    }
    red[w][lane] = acc;
    __syncthreads();
    if (w == 0 && d < D) partial2[nb * D + d] = red[0][lane] + red[1][lane] + red[2][lane] + red[3][lane];
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned total = gridDim.x * gridDim.y;
        last = atomicAdd(counter, 1u) == total - 1;
    }
    __syncthreads();
    if (!last) return;
    __threadfence();
    const int64_t nblk = gridDim.x;
    for (int64_t dd = threadIdx.x; dd < D; dd += blockDim.x) {
        double s = 0.0;
        for (int64_t k = 0; k < nblk; ++k) s += partial2[k * D + dd];
        double lv = (double)lam[dd];
        double sig = 1.0 / (1.0 + exp(-lv));
        dlambda[dd] = (float)(sig * s);
    }
    if (threadIdx.x == 0) *counter = 0u;
}

__global__ void fill_kernel(float* __restrict__ dst, float v, int64_t n) {
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) dst[i] = v;
}

hipError_t launch_fill(float* dst, float value, int64_t n, hipStream_t stream) {
    if (n <= 0 || dst == nullptr) return hipSuccess;
    hipLaunchKernelGGL(fill_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, dst,
                       value, n);
    return hipGetLastError();
}

size_t scan_backward_workspace(int64_t B, int64_t L, int64_t D, IoType) {
    (void)L;
    return bwd_ws_bytes(B, D);
}

template <typename T, typename TZ, int W, int C>
static hipError_t launch_bwd_chain(const ScanBwdArgs& a, hipStream_t stream) {
    const int64_t nch = a.B * a.D;
    BwdWorkspace ws = bwd_ws_carve(a.ws, a.B, a.D);
    dim3 grid((unsigned)((nch + kWave - 1) / kWave));
    if ((uint64_t)(nch * a.L) * sizeof(TZ) < (1ull << 32))
        hipLaunchKernelGGL((scan_bwd_chain_kernel<T, TZ, W, C, uint32_t>), grid, dim3(W * kWave),
                           0, stream, (const T*)a.x, (const TZ*)a.zr, (const TZ*)a.zi, a.lambda,
                           a.h0, (const T*)a.h, (const T*)a.dh, a.dhT, (T*)a.dx, (TZ*)a.dzr,
                           (TZ*)a.dzi, a.dh0, ws.partial, ws.counter, a.L, a.D, nch);
    else
        hipLaunchKernelGGL((scan_bwd_chain_kernel<T, TZ, W, C, uint64_t>), grid, dim3(W * kWave),
                           0, stream, (const T*)a.x, (const TZ*)a.zr, (const TZ*)a.zi, a.lambda,
                           a.h0, (const T*)a.h, (const T*)a.dh, a.dhT, (T*)a.dx, (TZ*)a.dzr,
                           (TZ*)a.dzi, a.dh0, ws.partial, ws.counter, a.L, a.D, nch);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    dim3 rgrid((unsigned)((a.B + kReduceRows - 1) / kReduceRows),
               (unsigned)((a.D + kWave - 1) / kWave));
    hipLaunchKernelGGL(dlambda_reduce_kernel, rgrid, dim3(256), 0, stream, ws.partial,
                       ws.partial2, ws.counter, a.lambda, a.dlambda, a.B, a.D);
    return hipGetLastError();
}

hipError_t launch_scan_backward(const ScanBwdArgs& a, hipStream_t stream) {
    if (a.io == IoType::kF32) return launch_bwd_chain<float, float, 8, 8>(a, stream);
    if (a.zio == IoType::kF32) return launch_bwd_chain<bf16, float, 8, 8>(a, stream);
    return launch_bwd_chain<bf16, bf16, 8, 8>(a, stream);
}

}  // namespace recblr
