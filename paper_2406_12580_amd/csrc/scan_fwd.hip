// Forward BD-LRU scan for gfx950: gate activation fused into the load,
// chunked along the sequence, carries combined through LDS.
//
// Recurrence (RecBLR, arXiv 2406.12580, eq:linrnn):  h_t = alpha_t h_{t-1} + beta'_t,
// beta'_t = beta_t x_t, with alpha, beta from the gate equations of section 3.2.
// The parallel form follows section 3.3: every segment of steps is an (A, H)
// pair, pairs compose with the associative operator "bullet", and the state at
// any step is the composition of all earlier segments applied to h0.
//
// Work decomposition ("chain" kernel):
//   * one lane owns one channel (b, d); the 64 lanes of a wave own 64
//     consecutive flattened channels c = b*D + d, so every load and store of
//     a time step is one contiguous run of 64 elements;
//   * a workgroup of W waves owns those 64 channels for the whole sequence and
//     walks it in macro-chunks of W*C steps; wave w scans steps
//     [w*C, w*C + C) of the macro-chunk sequentially in registers;
//   * the W wave aggregates (A, H) go through LDS; every wave folds the ones
//     before it onto the carry, re-runs its C steps from there and stores h;
//   * the carry after the macro-chunk stays in registers for the next one,
//     whose loads are already in flight (register double buffer).
// Each input element is read once and each output element written once.
#include "device_common.hpp"
#include "launch.hpp"

namespace recblr {

template <typename T, typename TZ, int C, bool RAW, typename Off>
struct ChunkRegs {
    float v0[C], v1[C], v2[C];  // gated: x, z_r, z_i;  raw: a, u (v2 unused)

    // Loads steps [t_first, t_first + C); steps past the end re-read step L-1
    // (always in bounds) and are masked by the caller.
    __device__ __forceinline__ void fetch(const T* __restrict__ p0, const TZ* __restrict__ p1,
                                          const TZ* __restrict__ p2, Off base, Off row,
                                          int64_t t_first, int64_t L) {
#pragma unroll
        for (int j = 0; j < C; ++j) {
            int64_t t = t_first + j < L ? t_first + j : L - 1;
            Off off = base + (Off)t * row;
            v0[j] = load_at(p0, off);
            v1[j] = load_at(p1, z_offset<T, TZ>(off));
            if (!RAW) v2[j] = load_at(p2, z_offset<T, TZ>(off));
        }
    }
};

template <typename T, typename TZ, int W, int C, bool RAW, typename Off>
__global__ __launch_bounds__(W* kWave) void scan_fwd_chain_kernel(
    const T* __restrict__ p0, const TZ* __restrict__ p1, const TZ* __restrict__ p2,
    const float* __restrict__ lam, const float* __restrict__ h0, T* __restrict__ h,
    float* __restrict__ hT, int64_t L, int64_t D, int64_t nch) {
    __shared__ Seg agg[2][W][kWave];
    const int lane = threadIdx.x & (kWave - 1);
    const int w = threadIdx.x / kWave;
    const int64_t c = (int64_t)blockIdx.x * kWave + lane;
    const bool valid = c < nch;
    const int64_t cs = valid ? c : 0;  // idle lanes shadow channel 0 and store nothing
    const int64_t b = cs / D;
    const int64_t d = cs - b * D;
    const Off base = (Off)((b * L * D + d) * (int64_t)sizeof(T));
    const Off row = (Off)(D * (int64_t)sizeof(T));
    ChannelConst cc{};
    if (!RAW) cc = channel_const(lam[d]);
    float carry = (valid && h0) ? h0[cs] : 0.0f;

    constexpr int64_t kMacro = (int64_t)W * C;
    ChunkRegs<T, TZ, C, RAW, Off> cur, nxt;
    if (L > 0) cur.fetch(p0, p1, p2, base, row, (int64_t)w * C, L);
    int buf = 0;
    for (int64_t t0 = 0; t0 < L; t0 += kMacro, buf ^= 1) {
        const int64_t tw = t0 + (int64_t)w * C;
        if (t0 + kMacro < L) nxt.fetch(p0, p1, p2, base, row, tw + kMacro, L);

        float a[C], u[C];
#pragma unroll
        for (int j = 0; j < C; ++j) {
            bool ok = (tw + j) < L;
            float aj, uj;
            if (RAW) {
                aj = cur.v0[j];
                uj = cur.v1[j];
            } else {
                gate_forward(cur.v0[j], cur.v1[j], cur.v2[j], cc, aj, uj);
            }
            a[j] = ok ? aj : 1.0f;  // steps past the end are the identity (1, 0)
            u[j] = ok ? uj : 0.0f;
        }
        // Local aggregate of this wave's C steps.
        Seg s{1.0f, 0.0f};
#pragma unroll
        for (int j = 0; j < C; ++j) s = compose(Seg{a[j], u[j]}, s);
        agg[buf][w][lane] = s;
        __syncthreads();

        // Carry into this wave: fold the aggregates of the earlier waves.
        float cin = carry;
#pragma unroll
        for (int k = 0; k < W; ++k) {
            if (k < w) {
                Seg e = agg[buf][k][lane];
                cin = fmaf(e.A, cin, e.H);
            }
        }
        // Re-run the C steps from the true carry and store h.
        float hv = cin;
#pragma unroll
        for (int j = 0; j < C; ++j) {
            hv = fmaf(a[j], hv, u[j]);
            if (valid && (tw + j) < L) store_at(h, base + (Off)(tw + j) * row, hv);
        }
        // Carry out of the macro-chunk: continue the fold through the last wave.
        float cout = cin;
#pragma unroll
        for (int k = 0; k < W; ++k) {
            if (k >= w) {
                Seg e = agg[buf][k][lane];
                cout = fmaf(e.A, cout, e.H);
            }
        }
        carry = cout;
        cur = nxt;
    }
    if (w == 0 && valid && hT) hT[cs] = carry;
}

// Copy h0 (or zeros) into hT: the L = 0 case.
__global__ void copy_state_kernel(const float* __restrict__ src, float* __restrict__ dst,
                                  int64_t n) {
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) dst[i] = src ? src[i] : 0.0f;
}

template <typename T, typename TZ, int W, int C, bool RAW>
static hipError_t launch_chain(const void* p0, const void* p1, const void* p2, const float* lam,
                               const float* h0, void* h, float* hT, int64_t B, int64_t L,
                               int64_t D, hipStream_t stream) {
    int64_t nch = B * D;
    dim3 grid((unsigned)((nch + kWave - 1) / kWave));
    // 32-bit byte offsets whenever a whole [B, L, D] tensor spans less than 4 GiB.
    if ((uint64_t)(nch * L) * sizeof(TZ) < (1ull << 32))
        hipLaunchKernelGGL((scan_fwd_chain_kernel<T, TZ, W, C, RAW, uint32_t>), grid,
                           dim3(W * kWave), 0, stream, (const T*)p0, (const TZ*)p1,
                           (const TZ*)p2, lam, h0, (T*)h, hT, L, D, nch);
    else
        hipLaunchKernelGGL((scan_fwd_chain_kernel<T, TZ, W, C, RAW, uint64_t>), grid,
                           dim3(W * kWave), 0, stream, (const T*)p0, (const TZ*)p1,
                           (const TZ*)p2, lam, h0, (T*)h, hT, L, D, nch);
    return hipGetLastError();
}

hipError_t launch_copy_state(const float* src, float* dst, int64_t n, hipStream_t stream) {
    if (n <= 0 || dst == nullptr) return hipSuccess;
    hipLaunchKernelGGL(copy_state_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0,
                       stream, src, dst, n);
    return hipGetLastError();
}

size_t scan_forward_workspace(int64_t, int64_t, int64_t, IoType) { return 0; }

hipError_t launch_scan_forward(const ScanFwdArgs& a, hipStream_t stream) {
    if (a.io == IoType::kF32)
        return launch_chain<float, float, 8, 8, false>(a.x, a.zr, a.zi, a.lambda, a.h0, a.h,
                                                       a.hT, a.B, a.L, a.D, stream);
    if (a.zio == IoType::kF32)
        return launch_chain<bf16, float, 8, 8, false>(a.x, a.zr, a.zi, a.lambda, a.h0, a.h, a.hT,
                                                      a.B, a.L, a.D, stream);
    return launch_chain<bf16, bf16, 8, 8, false>(a.x, a.zr, a.zi, a.lambda, a.h0, a.h, a.hT,
                                                 a.B, a.L, a.D, stream);
}

hipError_t launch_linear_scan(const float* a, const float* u, const float* h0, float* h,
                              float* hT, int64_t B, int64_t L, int64_t D, hipStream_t stream) {
    return launch_chain<float, float, 8, 8, true>(a, u, nullptr, nullptr, h0, h, hT, B, L, D,
                                                  stream);
}

}  // namespace recblr
