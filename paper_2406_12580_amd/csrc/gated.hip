// Gated recurrent layer core of RecBLR (arXiv 2406.12580, Algorithm
// alg:gated_recurrent: conv + SiLU, BD-LRU, output gate) outside the fused scan: the causal
// depthwise Conv1d + SiLU that forms the BD-LRU input, and the output gate
// y = h * SiLU(hz).  The scan kernel with the projections fused in applies
// the gate on the fly; these kernels serve the shapes it does not cover.
//
// Backward (the paper gives none; exact chain rule through the three lines):
//   dh = dy SiLU(hz),  dhz = dy h SiLU'(hz),  SiLU'(v) = s (1 + v (1 - s)), s = sigma(v)
//   (BD-LRU backward with projections at x' gives dx')
//   dc_t = dx'_t SiLU'(c_t),  dhx_t = sum_{j<K, t+j<L} w_j dc_{t+j}
//   dw_j = sum_{b, t>=j} dc_t hx_{t-j},  db = sum_{b,t} dc_t
#include "device_common.hpp"
#include "launch.hpp"

namespace recblr {
typedef uint32_t NtU4 __attribute__((ext_vector_type(4)));  // nontemporal 16-byte accesses

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

// x'_t = SiLU(b + sum_j w_j hx_{t-j}) with hx_{t<0} = 0, one element per
// thread; x' is stored as TO (the I/O type, or fp32 for a backward).
template <typename T, typename TO>
__global__ __launch_bounds__(kGateThreads) void conv_silu_kernel(const T* __restrict__ hx,
                                                                 const float* __restrict__ w4,
                                                                 const float* __restrict__ b4,
                                                                 TO* __restrict__ xp, int64_t L,
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

// The same with 16-byte loads (D % V == 0, 16-byte aligned tensors), each
// thread on kConvRun consecutive steps of one vector of V = 16 / sizeof(T)
// channels: every hx row it needs is loaded once and slides
// through registers (kConvRun + 3 row loads for kConvRun outputs instead of
// 4 per output).  Threads of a wave take consecutive channel vectors of the
// same rows.
constexpr int kConvRun = 4;  // 2 and 8 measured slower or no faster on the c4 / c5 shapes
template <typename T, typename TO>
__global__ __launch_bounds__(kGateThreads) void conv_silu_run_kernel(
    const T* __restrict__ hx, const float* __restrict__ w4, const float* __restrict__ b4,
    TO* __restrict__ xp, int64_t L, int64_t D, int64_t nthreads) {
    constexpr int V = 16 / sizeof(T);
    constexpr int VO = 16 / sizeof(TO);  // outputs per 16-byte store
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= nthreads) return;
    const int64_t dv = D / V, nrun = (L + kConvRun - 1) / kConvRun;
    const int64_t vec = q % dv, rest = q / dv;
    const int64_t run = rest % nrun, b = rest / nrun;
    const int64_t d = vec * V, t0 = run * kConvRun;
    float w[kConvTaps][V], bias[V];
#pragma unroll
    for (int i = 0; i < V; ++i) {
        bias[i] = b4[d + i];
#pragma unroll
        for (int j = 0; j < kConvTaps; ++j) w[j][i] = w4[j * D + d + i];
    }
    const T* row0 = hx + b * L * D + d;  // (b, 0, d)
    // win[j] = hx at step t - j (zero before the sequence start)
    float win[kConvTaps][V];
    // Every row the run needs is loaded before its first store, with no
    // branch around the loads (rows before 0 read row 0 and count as zero,
    // rows past L repeat row L - 1 and are not stored): vector memory
    // operations complete in issue order, so a load issued after a store
    // would be waited for together with it.
    uint4 halo[kConvTaps - 1], rows[kConvRun];
#pragma unroll
    for (int j = 1; j < kConvTaps; ++j) {
        const int64_t t = t0 - j;
        halo[j - 1] = *(const uint4*)(row0 + (t >= 0 ? t : 0) * D);
    }
#pragma unroll
    for (int s = 0; s < kConvRun; ++s) {
        const int64_t t = t0 + s < L ? t0 + s : L - 1;
        rows[s] = *(const uint4*)(row0 + t * D);
    }
#pragma unroll
    for (int j = 1; j < kConvTaps; ++j) {
        const T* v = (const T*)&halo[j - 1];
        const bool in = t0 - j >= 0;
#pragma unroll
        for (int i = 0; i < V; ++i) win[j][i] = in ? to_f32(v[i]) : 0.0f;
    }
#pragma unroll
    for (int s = 0; s < kConvRun; ++s) {
        const int64_t t = t0 + s;
        {
            const T* v = (const T*)&rows[s];
#pragma unroll
            for (int i = 0; i < V; ++i) win[0][i] = to_f32(v[i]);
        }
        float c[V];
#pragma unroll
        for (int i = 0; i < V; ++i) {
            float acc = bias[i];
#pragma unroll
            for (int j = 0; j < kConvTaps; ++j) acc = fmaf(w[j][i], win[j][i], acc);
            c[i] = acc;
        }
        TO* dst = xp + (b * L + t) * D + d;
#pragma unroll
        for (int s0 = 0; s0 < V; s0 += VO) {
            uint4 out;
            TO* o = (TO*)&out;
#pragma unroll
            for (int i = 0; i < VO; ++i) o[i] = from_f32<TO>(c[s0 + i] * sigmoid(c[s0 + i]));
            // (a plain store: x' is read again by the next kernels; a
            // nontemporal one measured 82 -> 130 us at 16 x 16384 x 256)
            if (t < L) *(uint4*)(dst + s0) = out;
        }
#pragma unroll
        for (int j = kConvTaps - 1; j > 0; --j)
#pragma unroll
            for (int i = 0; i < V; ++i) win[j][i] = win[j - 1][i];
    }
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

// ------------------------------------------------------------------ backward
__device__ __forceinline__ float dsilu(float v, float s) { return s * fmaf(v, 1.0f - s, 1.0f); }

// dh = dy SiLU(hz) and dhz = dy h SiLU'(hz), one element per thread; dh is
// stored as TG (fp32 when it feeds an fp32 backward), or not at all when dh
// is null (the fused scan then forms it on load).
template <typename T, typename TG>
__global__ __launch_bounds__(kGateThreads) void gate_bwd_kernel(
    const T* __restrict__ dy, const T* __restrict__ hz, const T* __restrict__ h,
    TG* __restrict__ dh, T* __restrict__ dhz, int64_t n) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= n) return;
    const float g = load(hz + e), s = sigmoid(g), gy = load(dy + e);
    if (dh) store(dh + e, gy * (g * s));
    store(dhz + e, gy * load(h + e) * dsilu(g, s));
}

// The same with 16-byte loads (n % V == 0, 16-byte aligned tensors).
template <typename T, typename TG>
__global__ __launch_bounds__(kGateThreads) void gate_bwd_vec_kernel(
    const T* __restrict__ dy, const T* __restrict__ hz, const T* __restrict__ h,
    TG* __restrict__ dh, T* __restrict__ dhz, int64_t nvec) {
    constexpr int V = 16 / sizeof(T);
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= nvec) return;
    // Streamed once: nontemporal loads and store (16 x 16384 x 256 bf16:
    // 106 -> 77 us).
    const uint4 ry = __builtin_bit_cast(uint4, __builtin_nontemporal_load((const NtU4*)(dy + q * V))),
                rz = __builtin_bit_cast(uint4, __builtin_nontemporal_load((const NtU4*)(hz + q * V))),
                rh = __builtin_bit_cast(uint4, __builtin_nontemporal_load((const NtU4*)(h + q * V)));
    const T* vy = (const T*)&ry;
    const T* vz = (const T*)&rz;
    const T* vh = (const T*)&rh;
    float g1[V];
    uint4 o2;
    T* b = (T*)&o2;
#pragma unroll
    for (int i = 0; i < V; ++i) {
        const float g = to_f32(vz[i]), s = sigmoid(g), gy = to_f32(vy[i]);
        g1[i] = gy * (g * s);
        b[i] = from_f32<T>(gy * to_f32(vh[i]) * dsilu(g, s));
    }
    constexpr int VG = 16 / sizeof(TG);
    if (dh) {
#pragma unroll
        for (int s0 = 0; s0 < V; s0 += VG) {
            uint4 o1;
            TG* a = (TG*)&o1;
#pragma unroll
            for (int i = 0; i < VG; ++i) a[i] = from_f32<TG>(g1[s0 + i]);
            *(uint4*)(dh + q * V + s0) = o1;
        }
    }
    __builtin_nontemporal_store(__builtin_bit_cast(NtU4, o2), (NtU4*)(dhz + q * V));
}

// bf16 to fp32, 8 elements per thread (n % 8 == 0, 16-byte aligned) or one.
__global__ __launch_bounds__(kGateThreads) void widen_kernel(const bf16* __restrict__ src,
                                                             float* __restrict__ dst, int64_t n,
                                                             bool vec) {
    const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (vec) {
        if (q * 8 >= n) return;
        const uint4 raw = *(const uint4*)(src + q * 8);
        const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
        float4 lo, hi;
        lo.x = bf16_lo(w[0]); lo.y = bf16_hi(w[0]); lo.z = bf16_lo(w[1]); lo.w = bf16_hi(w[1]);
        hi.x = bf16_lo(w[2]); hi.y = bf16_hi(w[2]); hi.z = bf16_lo(w[3]); hi.w = bf16_hi(w[3]);
        *(float4*)(dst + q * 8) = lo;
        *(float4*)(dst + q * 8 + 4) = hi;
    } else if (q < n) {
        dst[q] = to_f32(src[q]);
    }
}

// Conv backward (dx' of type TG: the I/O type or fp32).  A workgroup is 4 waves; lane l of wave w owns VEC channels
// d0 = (blockIdx.y * 64 + l) * VEC of batch row b and the chunk of kConvChunk
// steps number 4 * cg + w, with blockIdx.x = b * groups + cg.  The lane walks
// its chunk and the 3 steps after it (whose dc its last outputs need):
// it rebuilds c_t from hx with a 3-step window, forms dc_t, emits
// dhx_{t-3} = sum_j w_j dc_{t-3+j} from a 4-step window of dc (dc = 0 past
// L), and sums dc_t hx_{t-j} and dc_t over its own steps.  The 4 waves' sums
// are added in wave order and written as one row of partial[row][5][D]
// (taps 0..3, then the bias), row = blockIdx.x.
constexpr int kConvChunk = 64;
constexpr int kConvRowCols = kConvTaps + 1;

template <typename T, typename TG, int VEC>
__global__ __launch_bounds__(256) void conv_bwd_kernel(
    const T* __restrict__ hx, const TG* __restrict__ dxp, const float* __restrict__ w4,
    const float* __restrict__ b4, T* __restrict__ dhx, float* __restrict__ partial, int64_t L,
    int64_t D, int64_t groups) {
    __shared__ float red[4][kConvRowCols][kWave][VEC];
    const int lane = threadIdx.x & (kWave - 1), w = wave_id();
    const int64_t b = blockIdx.x / groups, cg = blockIdx.x - b * groups;
    const int64_t d0 = ((int64_t)blockIdx.y * kWave + lane) * VEC;
    const bool valid = d0 < D;
    const int64_t dc0 = valid ? d0 : 0;  // idle lanes shadow channel 0 and store nothing
    const int64_t t0 = (4 * cg + w) * kConvChunk;
    const int64_t end = t0 + kConvChunk < L ? t0 + kConvChunk : L;  // may be <= t0
    const int64_t tend = end + 3 < L ? end + 3 : L;
    float wt[kConvTaps][VEC], bias[VEC];
#pragma unroll
    for (int k = 0; k < VEC; ++k) {
        bias[k] = b4[dc0 + k];
#pragma unroll
        for (int j = 0; j < kConvTaps; ++j) wt[j][k] = w4[j * D + dc0 + k];
    }
    const int64_t rowb = b * L * D + dc0;  // element offset of (b, 0, d0)
    float h1[VEC], h2[VEC], h3[VEC];         // hx at t-1, t-2, t-3
    float e0[VEC], e1[VEC], e2[VEC], e3[VEC];  // dc at t, t-1, t-2, t-3
    float sw[kConvTaps][VEC], sb[VEC];
#pragma unroll
    for (int k = 0; k < VEC; ++k) {
        h1[k] = h2[k] = h3[k] = 0.0f;
        e0[k] = e1[k] = e2[k] = e3[k] = 0.0f;
        sb[k] = 0.0f;
#pragma unroll
        for (int j = 0; j < kConvTaps; ++j) sw[j][k] = 0.0f;
    }
    if (t0 < end) {
        if (t0 >= 3) load_vec<T, VEC>(hx, (rowb + (t0 - 3) * D) * (int64_t)sizeof(T), h3);
        if (t0 >= 2) load_vec<T, VEC>(hx, (rowb + (t0 - 2) * D) * (int64_t)sizeof(T), h2);
        if (t0 >= 1) load_vec<T, VEC>(hx, (rowb + (t0 - 1) * D) * (int64_t)sizeof(T), h1);
        // Unrolled for fp32 inputs, whose loads then overlap across steps
        // (c4-shaped backward 1414 -> 1365 us); bf16 measured slower unrolled.
#pragma unroll(sizeof(T) == 4 ? 4 : 1)
        for (int64_t t = t0; t < end + 3; ++t) {
            float dcv[VEC], x0[VEC];
            if (t < tend) {
                float g[VEC];
                load_vec<T, VEC>(hx, (rowb + t * D) * (int64_t)sizeof(T), x0);
                load_vec<TG, VEC>(dxp, (rowb + t * D) * (int64_t)sizeof(TG), g);
#pragma unroll
                for (int k = 0; k < VEC; ++k) {
                    float c = bias[k];
                    c = fmaf(wt[0][k], x0[k], c);
                    c = fmaf(wt[1][k], h1[k], c);
                    c = fmaf(wt[2][k], h2[k], c);
                    c = fmaf(wt[3][k], h3[k], c);
                    dcv[k] = g[k] * dsilu(c, sigmoid(c));
                }
                if (t < end) {
#pragma unroll
                    for (int k = 0; k < VEC; ++k) {
                        sb[k] += dcv[k];
                        sw[0][k] = fmaf(dcv[k], x0[k], sw[0][k]);
                        sw[1][k] = fmaf(dcv[k], h1[k], sw[1][k]);
                        sw[2][k] = fmaf(dcv[k], h2[k], sw[2][k]);
                        sw[3][k] = fmaf(dcv[k], h3[k], sw[3][k]);
                    }
                }
            } else {
#pragma unroll
                for (int k = 0; k < VEC; ++k) dcv[k] = x0[k] = 0.0f;
            }
#pragma unroll
            for (int k = 0; k < VEC; ++k) {
                e3[k] = e2[k];
                e2[k] = e1[k];
                e1[k] = e0[k];
                e0[k] = dcv[k];
                h3[k] = h2[k];
                h2[k] = h1[k];
                h1[k] = x0[k];
            }
            if (t - 3 >= t0 && valid) {
                float o[VEC];
#pragma unroll
                for (int k = 0; k < VEC; ++k)
                    o[k] = fmaf(wt[0][k], e3[k],
                                fmaf(wt[1][k], e2[k], fmaf(wt[2][k], e1[k], wt[3][k] * e0[k])));
                store_vec<T, VEC>(dhx, (rowb + (t - 3) * D) * (int64_t)sizeof(T), o);
            }
        }
    }
#pragma unroll
    for (int k = 0; k < VEC; ++k) {
#pragma unroll
        for (int j = 0; j < kConvTaps; ++j) red[w][j][lane][k] = sw[j][k];
        red[w][kConvTaps][lane][k] = sb[k];
    }
    __syncthreads();
    if (w == 0 && valid) {
        float* row = partial + (int64_t)blockIdx.x * kConvRowCols * D + dc0;
#pragma unroll
        for (int j = 0; j < kConvRowCols; ++j)
#pragma unroll
            for (int k = 0; k < VEC; ++k)
                row[j * D + k] = red[0][j][lane][k] + red[1][j][lane][k] + red[2][j][lane][k] +
                                 red[3][j][lane][k];
    }
}

// The same conv backward, software-pipelined: a lane's steps t0 .. end + 2
// run in blocks of kConvBlk, the loads of block j + 1 issued before the
// stores of block j (vector memory operations complete in issue order, so a
// load issued after a store is waited for together with it).  Every block
// issues the same operations: loads through per-row buffer resources at
// rows clamped to tend - 1 (values past tend taken as zero), stores of dhx
// at an offset past the resource where they must not land (the chunk's
// first three steps, steps past end + 2, idle lanes); the compiler's
// vector-memory wait counts are then exact.  Steps are processed in the
// order and with the arithmetic of conv_bwd_kernel, so the results are the
// same bit for bit.  Taken when a batch row of hx spans less than 2 GiB.
constexpr int kConvBlk = 4;
constexpr uint32_t kConvOOB = 0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t conv_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes,
                                             0x00020000);
}

// Cache policy of the buffer accesses: nontemporal (the tensors are streamed
// once; with the default policy the column sums that read the partials
// next took 21-27 instead of 17 us).
constexpr int kConvCP = 2;

template <typename T, int VEC>
__device__ __forceinline__ void conv_bload(__amdgpu_buffer_rsrc_t r, uint32_t off,
                                           float (&out)[VEC]) {
    static_assert(VEC == 1 || VEC == 4, "one or four channels per lane");
    if constexpr (sizeof(T) == 4) {
        if constexpr (VEC == 4) {
            typedef uint32_t u4 __attribute__((ext_vector_type(4)));
            const u4 v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kConvCP);
#pragma unroll
            for (int k = 0; k < 4; ++k) out[k] = __uint_as_float(v[k]);
        } else {
            out[0] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kConvCP));
        }
    } else {
        if constexpr (VEC == 4) {
            typedef uint32_t u2 __attribute__((ext_vector_type(2)));
            const u2 v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, kConvCP);
            out[0] = bf16_lo(v[0]);
            out[1] = bf16_hi(v[0]);
            out[2] = bf16_lo(v[1]);
            out[3] = bf16_hi(v[1]);
        } else {
            out[0] = __uint_as_float((uint32_t)__builtin_amdgcn_raw_buffer_load_b16(r, off, 0, kConvCP)
                                     << 16);
        }
    }
}

template <typename T, int VEC>
__device__ __forceinline__ void conv_bstore(__amdgpu_buffer_rsrc_t r, uint32_t off,
                                            const float (&in)[VEC]) {
    if constexpr (sizeof(T) == 4) {
        if constexpr (VEC == 4) {
            typedef uint32_t u4 __attribute__((ext_vector_type(4)));
            const u4 v = {__float_as_uint(in[0]), __float_as_uint(in[1]), __float_as_uint(in[2]),
                          __float_as_uint(in[3])};
            __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, kConvCP);
        } else {
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(in[0]), r, off, 0, kConvCP);
        }
    } else {
        if constexpr (VEC == 4) {
            typedef uint32_t u2 __attribute__((ext_vector_type(2)));
            const u2 v = {bf16_pair(in[0], in[1]), bf16_pair(in[2], in[3])};
            __builtin_amdgcn_raw_buffer_store_b64(v, r, off, 0, kConvCP);
        } else {
            __builtin_amdgcn_raw_buffer_store_b16((unsigned short)from_f32<bf16>(in[0]).bits, r,
                                                  off, 0, kConvCP);
        }
    }
}

template <typename T, typename TG, int VEC>
__global__ __launch_bounds__(256) void conv_bwd_piped_kernel(
    const T* __restrict__ hx, const TG* __restrict__ dxp, const float* __restrict__ w4,
    const float* __restrict__ b4, T* __restrict__ dhx, float* __restrict__ partial, int64_t L,
    int64_t D, int64_t groups) {
    constexpr int S = kConvBlk;
    __shared__ float red[4][kConvRowCols][kWave][VEC];
    const int lane = threadIdx.x & (kWave - 1), w = wave_id();
    const int64_t b = blockIdx.x / groups, cg = blockIdx.x - b * groups;
    const int64_t d0 = ((int64_t)blockIdx.y * kWave + lane) * VEC;
    const bool valid = d0 < D;
    const int64_t dc0 = valid ? d0 : 0;  // idle lanes shadow channel 0 and store nothing
    const int64_t t0 = (4 * cg + w) * kConvChunk;
    const int64_t end = t0 + kConvChunk < L ? t0 + kConvChunk : L;  // may be <= t0
    const int64_t tend = end + 3 < L ? end + 3 : L;
    float wt[kConvTaps][VEC], bias[VEC];
#pragma unroll
    for (int k = 0; k < VEC; ++k) {
        bias[k] = b4[dc0 + k];
#pragma unroll
        for (int j = 0; j < kConvTaps; ++j) wt[j][k] = w4[j * D + dc0 + k];
    }
    const uint32_t row_elems = (uint32_t)(L * D);
    const __amdgpu_buffer_rsrc_t rx = conv_rsrc(hx + b * L * D, row_elems * (uint32_t)sizeof(T));
    const __amdgpu_buffer_rsrc_t rg =
        conv_rsrc(dxp + b * L * D, row_elems * (uint32_t)sizeof(TG));
    const __amdgpu_buffer_rsrc_t ro = conv_rsrc(dhx + b * L * D, row_elems * (uint32_t)sizeof(T));
    auto elem = [&](int64_t t) -> uint32_t { return (uint32_t)(t * D + dc0); };
    float h1[VEC], h2[VEC], h3[VEC];           // hx at t-1, t-2, t-3
    float e0[VEC], e1[VEC], e2[VEC], e3[VEC];  // dc at t, t-1, t-2, t-3
    float sw[kConvTaps][VEC], sb[VEC];
#pragma unroll
    for (int k = 0; k < VEC; ++k) {
        h1[k] = h2[k] = h3[k] = 0.0f;
        e0[k] = e1[k] = e2[k] = e3[k] = 0.0f;
        sb[k] = 0.0f;
#pragma unroll
        for (int j = 0; j < kConvTaps; ++j) sw[j][k] = 0.0f;
    }
    if (t0 < end) {
        if (t0 >= 3) conv_bload<T, VEC>(rx, elem(t0 - 3) * (uint32_t)sizeof(T), h3);
        if (t0 >= 2) conv_bload<T, VEC>(rx, elem(t0 - 2) * (uint32_t)sizeof(T), h2);
        if (t0 >= 1) conv_bload<T, VEC>(rx, elem(t0 - 1) * (uint32_t)sizeof(T), h1);
        const int64_t tstop = end + 3;
        const int nb = (int)((tstop - t0 + S - 1) / S);
        auto load_blk = [&](int64_t tb, float (&xv)[S][VEC], float (&gv)[S][VEC]) {
#pragma unroll
            for (int i = 0; i < S; ++i) {
                const int64_t t = tb + i < tend ? tb + i : tend - 1;
                conv_bload<T, VEC>(rx, elem(t) * (uint32_t)sizeof(T), xv[i]);
                conv_bload<TG, VEC>(rg, elem(t) * (uint32_t)sizeof(TG), gv[i]);
            }
        };
        auto proc_blk = [&](int64_t tb, const float (&xv)[S][VEC], const float (&gv)[S][VEC]) {
#pragma unroll
            for (int i = 0; i < S; ++i) {
                const int64_t t = tb + i;
                float dcv[VEC], x0[VEC];
                if (t < tend) {
#pragma unroll
                    for (int k = 0; k < VEC; ++k) {
                        x0[k] = xv[i][k];
                        float c = bias[k];
                        c = fmaf(wt[0][k], x0[k], c);
                        c = fmaf(wt[1][k], h1[k], c);
                        c = fmaf(wt[2][k], h2[k], c);
                        c = fmaf(wt[3][k], h3[k], c);
                        dcv[k] = gv[i][k] * dsilu(c, sigmoid(c));
                    }
                    if (t < end) {
#pragma unroll
                        for (int k = 0; k < VEC; ++k) {
                            sb[k] += dcv[k];
                            sw[0][k] = fmaf(dcv[k], x0[k], sw[0][k]);
                            sw[1][k] = fmaf(dcv[k], h1[k], sw[1][k]);
                            sw[2][k] = fmaf(dcv[k], h2[k], sw[2][k]);
                            sw[3][k] = fmaf(dcv[k], h3[k], sw[3][k]);
                        }
                    }
                } else {
#pragma unroll
                    for (int k = 0; k < VEC; ++k) dcv[k] = x0[k] = 0.0f;
                }
#pragma unroll
                for (int k = 0; k < VEC; ++k) {
                    e3[k] = e2[k];
                    e2[k] = e1[k];
                    e1[k] = e0[k];
                    e0[k] = dcv[k];
                    h3[k] = h2[k];
                    h2[k] = h1[k];
                    h1[k] = x0[k];
                }
                float o[VEC];
#pragma unroll
                for (int k = 0; k < VEC; ++k)
                    o[k] = fmaf(wt[0][k], e3[k],
                                fmaf(wt[1][k], e2[k], fmaf(wt[2][k], e1[k], wt[3][k] * e0[k])));
                const bool keep = valid && t - 3 >= t0 && t < tstop;
                conv_bstore<T, VEC>(ro, keep ? elem(t - 3) * (uint32_t)sizeof(T) : kConvOOB, o);
            }
        };
        float xa[S][VEC], ga[S][VEC], xb[S][VEC], gb[S][VEC];
        load_blk(t0, xa, ga);
        for (int j = 0; j < nb; j += 2) {
            load_blk(t0 + (int64_t)(j + 1) * S, xb, gb);
            proc_blk(t0 + (int64_t)j * S, xa, ga);
            if (j + 1 >= nb) break;
            load_blk(t0 + (int64_t)(j + 2) * S, xa, ga);
            proc_blk(t0 + (int64_t)(j + 1) * S, xb, gb);
        }
    }
#pragma unroll
    for (int k = 0; k < VEC; ++k) {
#pragma unroll
        for (int j = 0; j < kConvTaps; ++j) red[w][j][lane][k] = sw[j][k];
        red[w][kConvTaps][lane][k] = sb[k];
    }
    __syncthreads();
    if (w == 0 && valid) {
        float* row = partial + (int64_t)blockIdx.x * kConvRowCols * D + dc0;
#pragma unroll
        for (int j = 0; j < kConvRowCols; ++j)
#pragma unroll
            for (int k = 0; k < VEC; ++k)
                row[j * D + k] = red[0][j][lane][k] + red[1][j][lane][k] + red[2][j][lane][k] +
                                 red[3][j][lane][k];
    }
}

// Column sums of partial[rows][cols] in a fixed order, in double: block
// (nb, cb) adds rows [nb * 64, nb * 64 + 64) of columns [cb * 256, + 256).
constexpr int kColRows = 64;
__global__ __launch_bounds__(256) void colsum_rows_kernel(const float* __restrict__ partial,
                                                          double* __restrict__ part2,
                                                          int64_t rows, int64_t cols) {
    const int64_t col = (int64_t)blockIdx.y * 256 + threadIdx.x;
    if (col >= cols) return;
    const int64_t r0 = (int64_t)blockIdx.x * kColRows;
    const int64_t r1 = r0 + kColRows < rows ? r0 + kColRows : rows;
    double acc = 0.0;
    for (int64_t r = r0; r < r1; ++r) acc += (double)partial[r * cols + col];
    part2[(int64_t)blockIdx.x * cols + col] = acc;
}

// The row blocks added in order, then written as dconv_w[d][j] (j < K) and
// dconv_b[d] (if not null) from the columns [j][d] and [kConvTaps][d].
__global__ __launch_bounds__(256) void conv_grad_final_kernel(const double* __restrict__ part2,
                                                              int64_t nblk, int64_t D, int K,
                                                              float* __restrict__ dw,
                                                              float* __restrict__ db) {
    const int64_t col = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t cols = kConvRowCols * D;
    if (col >= cols) return;
    double acc = 0.0;
    for (int64_t r = 0; r < nblk; ++r) acc += part2[r * cols + col];
    const int64_t j = col / D, d = col - j * D;
    if (j < K) dw[d * K + j] = (float)acc;
    else if (j == kConvTaps && db) db[d] = (float)acc;
}

namespace {
template <typename T, typename TG>
hipError_t gate_backward_t(const void* dy, const void* hz, const void* h, void* dh, void* dhz,
                           int64_t n, hipStream_t stream) {
    constexpr int V = 16 / sizeof(T);
    if (n % V == 0 &&
        ((uintptr_t)dy | (uintptr_t)hz | (uintptr_t)h | (uintptr_t)dh | (uintptr_t)dhz) % 16 == 0) {
        const int64_t nvec = n / V;
        hipLaunchKernelGGL((gate_bwd_vec_kernel<T, TG>),
                           dim3((unsigned)((nvec + kGateThreads - 1) / kGateThreads)),
                           dim3(kGateThreads), 0, stream, (const T*)dy, (const T*)hz, (const T*)h,
                           (TG*)dh, (T*)dhz, nvec);
    } else {
        hipLaunchKernelGGL((gate_bwd_kernel<T, TG>),
                           dim3((unsigned)((n + kGateThreads - 1) / kGateThreads)),
                           dim3(kGateThreads), 0, stream, (const T*)dy, (const T*)hz, (const T*)h,
                           (TG*)dh, (T*)dhz, n);
    }
    return hipGetLastError();
}
}  // namespace

// Column sums of a tall [rows][cols] matrix, in a fixed order.  Stage 1:
// workgroup (b, tile) adds rows [b * R, b * R + R) of up to 256 columns; its
// 256 threads are J = 256 / tc row lanes of tc columns, lane j adding rows
// j, j + J, ... in double, and the J lanes are then added in lane order.
// Stage 2 adds the G workgroup sums of each column (colsum_short_kernel).
constexpr int kColsumGroups = 512;
__global__ __launch_bounds__(256) void colsum_part_kernel(const float* __restrict__ src,
                                                          double* __restrict__ part,
                                                          int64_t rows, int64_t cols,
                                                          int64_t rows_per_group) {
    __shared__ double sh[256];
    const int64_t tc = cols < 256 ? cols : 256;
    const int J = (int)(256 / tc);
    const int t = threadIdx.x;
    const int j = (int)(t / tc);
    const int64_t c = (int64_t)blockIdx.y * 256 + (t % tc);
    const int64_t r0 = (int64_t)blockIdx.x * rows_per_group;
    const int64_t r1 = r0 + rows_per_group < rows ? r0 + rows_per_group : rows;
    double acc = 0.0;
    if (j < J && c < cols) {
        // 8 loads in flight, added in row order
        int64_t r = r0 + j;
        for (; r + 7 * J < r1; r += 8 * J) {
            float v[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) v[q] = src[(r + q * J) * cols + c];
#pragma unroll
            for (int q = 0; q < 8; ++q) acc += (double)v[q];
        }
        for (; r < r1; r += J) acc += (double)src[r * cols + c];
    }
    sh[t] = acc;
    __syncthreads();
    if (j == 0 && c < cols) {
        double s = sh[t];
        for (int q = 1; q < J; ++q) s += sh[q * tc + t];
        part[(int64_t)blockIdx.x * cols + c] = s;
    }
}

// Column sums of a short matrix (rows <= kColsumGroups, the split partials of
// the weight gradients and the LayerNorm parameter gradients) in one launch:
// the four waves of a workgroup take four consecutive row ranges of the same
// 64 columns, each summed in row order in double (8 loads in flight), and the
// four range sums are added in range order.
template <typename TS>
__global__ __launch_bounds__(256) void colsum_short_kernel(const TS* __restrict__ src,
                                                           int64_t rows, int64_t cols,
                                                           float* __restrict__ out) {
    __shared__ double sh[4][64];
    const int lane = threadIdx.x & 63, q = threadIdx.x >> 6;
    const int64_t c = (int64_t)blockIdx.x * 64 + lane;
    const int64_t per = (rows + 3) / 4;
    const int64_t r0 = q * per, r1 = r0 + per < rows ? r0 + per : rows;
    double acc = 0.0;
    if (c < cols) {
        int64_t r = r0;
        for (; r + 8 <= r1; r += 8) {
            TS v[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) v[k] = src[(r + k) * cols + c];
#pragma unroll
            for (int k = 0; k < 8; ++k) acc += (double)v[k];
        }
        for (; r < r1; ++r) acc += (double)src[r * cols + c];
    }
    sh[q][lane] = acc;
    __syncthreads();
    if (q == 0 && c < cols)
        out[c] = (float)(((sh[0][lane] + sh[1][lane]) + sh[2][lane]) + sh[3][lane]);
}

size_t colsum_workspace(int64_t rows, int64_t cols) {
    const int64_t g = rows < kColsumGroups ? (rows > 0 ? rows : 1) : kColsumGroups;
    return (size_t)(g * cols) * sizeof(double);
}

hipError_t launch_colsum(const float* src, int64_t rows, int64_t cols, float* out, void* ws,
                         hipStream_t stream) {
    if (cols == 0) return hipSuccess;
    if (rows == 0) return launch_fill(out, 0.0f, cols, stream);
    if (rows <= kColsumGroups) {
        hipLaunchKernelGGL(colsum_short_kernel<float>, dim3((unsigned)((cols + 63) / 64)),
                           dim3(256), 0, stream, src, rows, cols, out);
        return hipGetLastError();
    }
    const int64_t groups = kColsumGroups;
    const int64_t per = (rows + groups - 1) / groups;
    double* part = (double*)ws;
    hipLaunchKernelGGL(colsum_part_kernel, dim3((unsigned)groups, (unsigned)((cols + 255) / 256)),
                       dim3(256), 0, stream, src, part, rows, cols, per);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // Stage 2: the group sums of each column, as a short matrix of doubles.
    hipLaunchKernelGGL(colsum_short_kernel<double>, dim3((unsigned)((cols + 63) / 64)), dim3(256),
                       0, stream, part, groups, cols, out);
    return hipGetLastError();
}

hipError_t launch_gate_backward(const void* dy, const void* hz, const void* h, void* dh,
                                void* dhz, int64_t n, IoType io, IoType dh_io,
                                hipStream_t stream) {
    if (n == 0) return hipSuccess;
    if (io == IoType::kF32) return gate_backward_t<float, float>(dy, hz, h, dh, dhz, n, stream);
    if (dh_io == IoType::kF32) return gate_backward_t<bf16, float>(dy, hz, h, dh, dhz, n, stream);
    return gate_backward_t<bf16, bf16>(dy, hz, h, dh, dhz, n, stream);
}

hipError_t launch_widen(const void* src, float* dst, int64_t n, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    const bool vec = n % 8 == 0 && ((uintptr_t)src | (uintptr_t)dst) % 16 == 0;
    const int64_t threads = vec ? n / 8 : n;
    hipLaunchKernelGGL(widen_kernel, dim3((unsigned)((threads + kGateThreads - 1) / kGateThreads)),
                       dim3(kGateThreads), 0, stream, (const bf16*)src, dst, n, vec);
    return hipGetLastError();
}

namespace {
struct ConvBwdPlan {
    int64_t groups;  // workgroups along the sequence per batch row (4 chunks each)
    int64_t rows;    // partial rows = B * groups
    int64_t nblk;    // row blocks of the column sums
    size_t partial_bytes, part2_bytes;
};
ConvBwdPlan conv_bwd_plan(int64_t B, int64_t L, int64_t D) {
    ConvBwdPlan p;
    const int64_t chunks = (L + kConvChunk - 1) / kConvChunk;
    p.groups = chunks > 0 ? (chunks + 3) / 4 : 1;
    p.rows = B * p.groups;
    p.nblk = (p.rows + kColRows - 1) / kColRows;
    p.partial_bytes = (size_t)(p.rows * kConvRowCols * D) * sizeof(float);
    p.part2_bytes = (size_t)(p.nblk * kConvRowCols * D) * sizeof(double);
    return p;
}
size_t align256(size_t v) { return (v + 255) / 256 * 256; }
}  // namespace

size_t conv_backward_workspace(int64_t B, int64_t L, int64_t D) {
    const ConvBwdPlan p = conv_bwd_plan(B, L, D);
    return align256(p.partial_bytes) + align256(p.part2_bytes);
}

namespace {
template <typename T, typename TG, int VEC>
void conv_backward_t(dim3 grid, const void* hx, const void* dxp, const float* w4, const float* b4,
                     void* dhx, float* partial, int64_t L, int64_t D, int64_t groups,
                     hipStream_t stream) {
    // The pipelined kernel addresses a batch row with 32-bit offsets.
    if (L * D * (int64_t)(sizeof(T) > sizeof(TG) ? sizeof(T) : sizeof(TG)) < ((int64_t)1 << 31))
        hipLaunchKernelGGL((conv_bwd_piped_kernel<T, TG, VEC>), grid, dim3(256), 0, stream,
                           (const T*)hx, (const TG*)dxp, w4, b4, (T*)dhx, partial, L, D, groups);
    else
        hipLaunchKernelGGL((conv_bwd_kernel<T, TG, VEC>), grid, dim3(256), 0, stream,
                           (const T*)hx, (const TG*)dxp, w4, b4, (T*)dhx, partial, L, D, groups);
}
}  // namespace

hipError_t launch_conv_backward(const void* hx, const void* dxp, const float* w4, const float* b4,
                                void* dhx, float* dw, float* db, int K, int64_t B, int64_t L,
                                int64_t D, IoType io, IoType dxp_io, void* ws,
                                hipStream_t stream) {
    const ConvBwdPlan p = conv_bwd_plan(B, L, D);
    float* partial = (float*)ws;
    double* part2 = (double*)((char*)ws + align256(p.partial_bytes));
    const uintptr_t amask = (uintptr_t)hx | (uintptr_t)dhx;
    const bool v4 = D % 4 == 0 && amask % (4 * io_bytes(io)) == 0 &&
                    (uintptr_t)dxp % (4 * io_bytes(dxp_io)) == 0;
    const dim3 grid((unsigned)(B * p.groups), (unsigned)((D / (v4 ? 4 : 1) + kWave - 1) / kWave));
    const bool g32 = dxp_io == IoType::kF32;
    if (io == IoType::kF32) {
        if (v4) conv_backward_t<float, float, 4>(grid, hx, dxp, w4, b4, dhx, partial, L, D, p.groups, stream);
        else conv_backward_t<float, float, 1>(grid, hx, dxp, w4, b4, dhx, partial, L, D, p.groups, stream);
    } else if (g32) {
        if (v4) conv_backward_t<bf16, float, 4>(grid, hx, dxp, w4, b4, dhx, partial, L, D, p.groups, stream);
        else conv_backward_t<bf16, float, 1>(grid, hx, dxp, w4, b4, dhx, partial, L, D, p.groups, stream);
    } else {
        if (v4) conv_backward_t<bf16, bf16, 4>(grid, hx, dxp, w4, b4, dhx, partial, L, D, p.groups, stream);
        else conv_backward_t<bf16, bf16, 1>(grid, hx, dxp, w4, b4, dhx, partial, L, D, p.groups, stream);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t cols = kConvRowCols * D;
    hipLaunchKernelGGL(colsum_rows_kernel, dim3((unsigned)p.nblk, (unsigned)((cols + 255) / 256)),
                       dim3(256), 0, stream, partial, part2, p.rows, cols);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(conv_grad_final_kernel, dim3((unsigned)((cols + 255) / 256)), dim3(256), 0,
                       stream, part2, p.nblk, D, K, dw, db);
    return hipGetLastError();
}

hipError_t launch_pack_conv(const float* w, const float* b, int K, int64_t D, float* w4,
                            float* b4, hipStream_t stream) {
    hipLaunchKernelGGL(pack_conv_kernel, dim3((unsigned)((D + 255) / 256)), dim3(256), 0, stream,
                       w, b, K, D, w4, b4);
    return hipGetLastError();
}

namespace {
template <typename T, typename TO>
hipError_t conv_silu_t(const void* hx, const float* w4, const float* b4, void* xp, int64_t L,
                       int64_t D, int64_t n, hipStream_t stream) {
    constexpr int V = 16 / sizeof(T);
    if (n == 0) return hipSuccess;
    if (D % V == 0 && ((uintptr_t)hx | (uintptr_t)xp) % 16 == 0) {
        const int64_t nthreads = (n / (L * D)) * ((L + kConvRun - 1) / kConvRun) * (D / V);
        hipLaunchKernelGGL((conv_silu_run_kernel<T, TO>),
                           dim3((unsigned)((nthreads + kGateThreads - 1) / kGateThreads)),
                           dim3(kGateThreads), 0, stream, (const T*)hx, w4, b4, (TO*)xp, L, D,
                           nthreads);
    } else {
        hipLaunchKernelGGL((conv_silu_kernel<T, TO>),
                           dim3((unsigned)((n + kGateThreads - 1) / kGateThreads)),
                           dim3(kGateThreads), 0, stream, (const T*)hx, w4, b4, (TO*)xp, L, D, n);
    }
    return hipGetLastError();
}
}  // namespace

hipError_t launch_conv_silu(const void* hx, const float* w4, const float* b4, void* xp, int64_t B,
                            int64_t L, int64_t D, IoType io, IoType out_io, hipStream_t stream) {
    const int64_t n = B * L * D;
    if (n == 0) return hipSuccess;
    if (io == IoType::kF32) return conv_silu_t<float, float>(hx, w4, b4, xp, L, D, n, stream);
    if (out_io == IoType::kF32) return conv_silu_t<bf16, float>(hx, w4, b4, xp, L, D, n, stream);
    return conv_silu_t<bf16, bf16>(hx, w4, b4, xp, L, D, n, stream);
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
