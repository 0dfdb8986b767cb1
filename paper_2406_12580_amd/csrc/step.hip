// One recurrent step of the BD-LRU for inference (RecBLR, arXiv 2406.12580,
// eq:linrnn with the gates of section 3.2):
//   h_next[b, d] = alpha(z_r) h_prev[b, d] + beta(z_r, z_i) x[b, d]
// Purely elementwise and bound by HBM bandwidth.  Each thread handles 8
// consecutive elements (one 16-byte bf16 load or two 16-byte fp32 loads per
// operand); the per-channel constants of softplus(Lambda) are built once per
// workgroup in LDS.
#include <type_traits>
#include <utility>

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
// One group of 8 elements per thread and no grid-stride loop: every thread
// issues its loads at once (a grid-stride loop over fewer workgroups measured
// 42-43 us against 40-40.5 us at 65536 x 256, bf16 with fp32 state).
template <typename T, typename TZ>
__global__ __launch_bounds__(kStepThreads) void step_vec_kernel(
    const T* __restrict__ x, const TZ* __restrict__ zr, const TZ* __restrict__ zi,
    const float* __restrict__ lam, const float* h_prev, float* h_next, int64_t n, int64_t D) {
    __shared__ ChannelConst table[kStepMaxTable];
    for (int64_t d = threadIdx.x; d < D; d += blockDim.x) table[d] = channel_const(lam[d]);
    __syncthreads();
    const int64_t e0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * kStepVec;
    if (e0 < n) {
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
        const int64_t blocks = (n / kStepVec + kStepThreads - 1) / kStepThreads;
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


// ----------------------------------------------------------------------------
// Recurrent step with the gate projections fused in, bf16 I/O, D = 64..256
// (D % 64 == 0):
//   z_r = W_r x + b_r, z_i = W_i x + b_i   (section 3.2), then the step above,
// with z kept in registers.
//
// Both weight matrices together are 2 D^2 bf16 (256 KB at D = 256): too much
// for LDS, but half of a compute unit's vector register file.  So each
// workgroup is persistent and keeps them resident: wave w of 2 D / 32 holds,
// as bf16 MFMA B-fragments, the rows of W_r and W_i of its 16 channels
// 16 w .. 16 w + 15 (8 D / 32 VGPRs per lane), and the workgroup then walks
// blocks of 16 batch rows.  A block's x rows (16 x D bf16) are staged in LDS
// and feed every wave's A-fragments; wave w's 16 x 16 product for each gate
// (v_mfma_f32_16x16x32_bf16, fp32 accumulation) leaves z_r, z_i of 4 rows of
// one channel in each lane, which reads h_prev and writes h_next there.
// Each block's global loads are issued two (h_prev) and four (x) blocks ahead
// of their use, and the matrix products of block k + 1 overlap the step of
// block k (see the pipeline below).  The kernel is bound by the issue of its
// vector, matrix and memory instructions between the per-block barriers: a
// copy of it without products and gate arithmetic streams the same bytes at
// 5.0 TB/s, the whole step at about 3.6 TB/s.
namespace resident {

typedef __bf16 b8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u2v __attribute__((ext_vector_type(2)));

constexpr int RB = 16;  // batch rows per block (one MFMA row tile)
constexpr uint32_t kOOB = 0x80000000u;  // past every resource: loads give 0, stores drop

__device__ __forceinline__ __amdgpu_buffer_rsrc_t resource(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes,
                                             0x00020000);
}

// LDS x block: rows of D bf16 padded by 16 bytes, so that a fragment read
// (16 rows, one 16-byte chunk each) falls on 16 distinct bank groups and every
// address a lane reads is its row base plus a constant.
template <int D>
constexpr int kPitch = 2 * D + 16;

template <int KS>
__global__ __launch_bounds__(128 * KS) void step_resident_kernel(
    const bf16* x, const bf16* wr, const bf16* wi, const bf16* br, const bf16* bi,
    const float* lam, const float* h_prev, float* h_next, int64_t B) {
    constexpr int D = 32 * KS;  // channels; K of the products
    constexpr int QPR = D / 4;  // 8-byte x quads per row
    constexpr int PITCH = kPitch<D>;
    __shared__ __attribute__((aligned(16))) char xs[3][RB * PITCH];
    const int tid = threadIdx.x, w = wave_id(), lane = tid & 63;
    const int fr = lane & 15, fq = lane >> 4;
    const int ch = 16 * w + fr;
    const ChannelConst cc = channel_const(lam[ch]);
    const float bzr = br ? to_f32(br[ch]) : 0.0f;
    const float bzi = bi ? to_f32(bi[ch]) : 0.0f;

    // This workgroup's blocks: g, g + G, g + 2 G, ... (k-th is g + k G).
    // Byte offsets are a wave-uniform block base (saturated at kOOB, so
    // blocks past the end read zeros and store nothing) plus a lane part;
    // rows past B fall outside the resources in the same way.
    const int64_t nblk = (B + RB - 1) / RB, G = gridDim.x, g = blockIdx.x;
    const int64_t nk = (nblk - g + G - 1) / G;
    const __amdgpu_buffer_rsrc_t rx = resource(x, (uint32_t)(B * D * 2));
    const __amdgpu_buffer_rsrc_t rh = resource(h_prev, (uint32_t)(B * D * 4));
    const __amdgpu_buffer_rsrc_t ro = resource(h_next, (uint32_t)(B * D * 4));
    auto base = [&](int64_t k, int esz) -> uint32_t {
        const int64_t o = (g + k * G) * RB * D * esz;
        return k < nk && o < (int64_t)kOOB ? (uint32_t)o : kOOB;
    };
    // x staging: thread tid moves quad (row tid / QPR, columns 4 (tid % QPR) .. + 3).
    const int sr = tid / QPR, sc = 4 * (tid % QPR);
    const int s_lds = sr * PITCH + 2 * sc;
    const uint32_t x_lane = (uint32_t)((sr * D + sc) * 2);
    auto x_off = [&](int64_t k) -> uint32_t { return base(k, 2) + x_lane; };
    // Rows of this lane's outputs in a block: 4 fq + v.
    const uint32_t h_lane = (uint32_t)((4 * fq * D + ch) * 4);
    auto h_off = [&](int64_t k, int v) -> uint32_t { return base(k, 4) + h_lane + v * D * 4; };
    const int a_lds = fr * PITCH + 16 * fq;    // fragment: row fr, chunk 4 kk + fq
    const int e_lds = 4 * fq * PITCH + 2 * ch;  // epilogue: row 4 fq + v, column ch

    // Software pipeline over this workgroup's blocks k = 0 .. nk-1, with
    // slot p = k mod 2 of the register buffers and LDS buffer k mod 3:
    //   MFMAs of block k + 1 (x rows already in LDS) into acc[1 - p], while
    //   the step of block k runs on acc[p] (the matrix cores and the vector
    //   ALUs overlap); then the h_prev loads of block k + 2 into hp[p], the
    //   x rows of block k + 2 from xq[p] into LDS, and the x loads of block
    //   k + 4 into xq[p].
    u2v xq[2];
    float hp[2][4];
    f4 acc[2][2];
    b8 wrf[KS], wif[KS];
    constexpr int BUF = RB * PITCH;
    char* const xs0 = &xs[0][0];
    auto mma = [&](int buf, f4 (&o)[2]) {
        const char* xb = xs0 + buf * BUF;
        f4 ar = {bzr, bzr, bzr, bzr}, ai = {bzi, bzi, bzi, bzi};
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) {
            const b8 fa = *(const b8*)&xb[a_lds + 64 * kk];
            ar = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa, wrf[kk], ar, 0, 0, 0);
            ai = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa, wif[kk], ai, 0, 0, 0);
        }
        o[0] = ar;
        o[1] = ai;
    };
    {
        const u2v x0 = __builtin_amdgcn_raw_buffer_load_b64(rx, x_off(0), 0, 0);
        const u2v x1 = __builtin_amdgcn_raw_buffer_load_b64(rx, x_off(1), 0, 0);
#pragma unroll
        for (int p = 0; p < 2; ++p) {
#pragma unroll
            for (int v = 0; v < 4; ++v)
                hp[p][v] =
                    __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rh, h_off(p, v), 0, 0));
            xq[p] = __builtin_amdgcn_raw_buffer_load_b64(rx, x_off(p + 2), 0, 0);
        }
        // Resident B-fragments: lane (fr, fq) holds W[ch][32 kk + 8 fq .. + 7].
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) {
            wrf[kk] = *(const b8*)(wr + (int64_t)ch * D + 32 * kk + 8 * fq);
            wif[kk] = *(const b8*)(wi + (int64_t)ch * D + 32 * kk + 8 * fq);
        }
        // Everything above lands before the pipeline starts, so that the
        // loop's waits count only the loop's own loads.
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
        __builtin_amdgcn_sched_barrier(0);
        *(u2v*)&xs0[s_lds] = x0;
        *(u2v*)&xs0[BUF + s_lds] = x1;
        __syncthreads();
        mma(0, acc[0]);
    }

    auto block = [&](int64_t k, int buf, auto slot) {
        constexpr int p = decltype(slot)::value;
        const int nbuf = buf == 2 ? 0 : buf + 1, fbuf = nbuf == 2 ? 0 : nbuf + 1;
        mma(nbuf, acc[1 - p]);
        const char* xb = xs0 + buf * BUF;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const uint32_t xbits = *(const uint16_t*)&xb[e_lds + v * PITCH];
            float a, u;
            gate_forward(__uint_as_float(xbits << 16), acc[p][0][v], acc[p][1][v], cc, a, u);
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(fmaf(a, hp[p][v], u)), ro,
                                                  h_off(k, v), 0, 0);
        }
#pragma unroll
        for (int v = 0; v < 4; ++v)
            hp[p][v] =
                __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rh, h_off(k + 2, v), 0, 0));
        *(u2v*)&xs0[fbuf * BUF + s_lds] = xq[p];
        xq[p] = __builtin_amdgcn_raw_buffer_load_b64(rx, x_off(k + 4), 0, 0);
        __syncthreads();
        return nbuf;
    };
    // Whole rounds of two blocks in the loop and the last odd block after
    // it, so that every path around the loop issues the same loads (the
    // compiler's wait counts then stay exact across the back edge).
    using S0 = std::integral_constant<int, 0>;
    using S1 = std::integral_constant<int, 1>;
    int64_t k = 0;
    int buf = 0;
    for (; k + 2 <= nk; k += 2) {
        buf = block(k, buf, S0{});
        buf = block(k + 1, buf, S1{});
    }
    if (k < nk) block(k, buf, S0{});
}

template <int KS>
int resident_grid(int64_t nblk) {
    static const int per_cu = [] {
        int n = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, step_resident_kernel<KS>,
                                                         128 * KS, 0) != hipSuccess || n < 1)
            n = 1;
        return n;
    }();
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus < 1)
        cus = 256;
    const int64_t g = (int64_t)cus * per_cu;
    return (int)(nblk < g ? nblk : g);
}

template <int KS>
hipError_t launch_ks(const void* x, const void* wr, const void* br, const void* wi,
                     const void* bi, const float* lam, const float* h_prev, float* h_next,
                     int64_t B, hipStream_t stream) {
    const int64_t nblk = (B + RB - 1) / RB;
    hipLaunchKernelGGL(step_resident_kernel<KS>, dim3((unsigned)resident_grid<KS>(nblk)),
                       dim3(128 * KS), 0, stream, (const bf16*)x, (const bf16*)wr,
                       (const bf16*)wi, (const bf16*)br, (const bf16*)bi, lam, h_prev, h_next, B);
    return hipGetLastError();
}

}  // namespace resident

bool launch_step_resident(const void* x, const void* wr, const void* br, const void* wi,
                          const void* bi, const float* lambda, const float* h_prev,
                          float* h_next, int64_t B, int64_t D, IoType io, hipStream_t stream,
                          hipError_t* err) {
    if (io != IoType::kBf16 || B <= 0 || D % 64 != 0 || D < 64 || D > 256 ||
        !aligned16(x) || !aligned16(wr) || !aligned16(wi) || B * D * 4 >= (int64_t)resident::kOOB)
        return false;
    switch (D) {
        case 64: *err = resident::launch_ks<2>(x, wr, br, wi, bi, lambda, h_prev, h_next, B, stream); break;
        case 128: *err = resident::launch_ks<4>(x, wr, br, wi, bi, lambda, h_prev, h_next, B, stream); break;
        case 192: *err = resident::launch_ks<6>(x, wr, br, wi, bi, lambda, h_prev, h_next, B, stream); break;
        default: *err = resident::launch_ks<8>(x, wr, br, wi, bi, lambda, h_prev, h_next, B, stream); break;
    }
    return true;
}

}  // namespace recblr
