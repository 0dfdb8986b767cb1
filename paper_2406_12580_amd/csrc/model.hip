// One training step of the full RecBLR model (arXiv 2406.12580): embedding
// with LayerNorm (section 2, eq:layernorm), `layers` behaviour-modelling
// layers (section 3.1: the gated recurrent layer of Algorithm
// alg:gated_recurrent, then the PFFN of eq. PFFN, each sub-layer followed by a
// residual connection and LayerNorm), and the prediction layer (section 2:
// softmax over h_T E^T) with the cross entropy of the next item; then Adam.
//
// The linear layers of the behaviour-modelling layers run on the matrix-core
// kernels of gemm.hip (fp32 MFMAs for forward products and data gradients,
// with the bias, SiLU and SiLU' in their epilogues; bf16-split tiles for the
// weight gradients); the prediction layer's products are rocBLAS fp32 GEMMs;
// everything else runs in the kernels of this library: the gated recurrent layer core through
// recblr_gated_forward / recblr_gated_backward (conv, BD-LRU scan with its
// gate projections, output gate), and here the embedding gather, the
// LayerNorms, bias broadcasts, SiLU, the cross entropy, the sums over rows
// for bias and LayerNorm gradients (fixed order, double), the embedding
// gradient (positions sorted by item, then summed per item in position
// order), the dropout masks (one bit per element from a counter-based
// generator, applied inside the LayerNorm kernels) and Adam.
#include <hip/hip_runtime.h>
#include <rocblas/rocblas.h>

#include <hipcub/hipcub.hpp>

#include "device_common.hpp"
#include "gemm.hpp"
#include "launch.hpp"
#include "model.hpp"
#include "recblr.h"

namespace recblr {
namespace model {

namespace {

constexpr int kThreads = 256;
constexpr int kLnRows = 4;  // rows each wave of the LayerNorm forward normalises together
constexpr int64_t kLnBwdRows = 256;  // rows per workgroup of the LayerNorm backward
constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// ------------------------------------------------------------------ dropout masks
// Philox4x64-10 (Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as
// easy as 1, 2, 3", SC 2011), in place on the counter c under key (k0, k1):
// ten rounds, each multiplying words 0 and 2 by the round multipliers and
// mixing the product halves with words 1 and 3 and the key; the key is
// bumped by the Weyl constants between rounds.
// The 128-bit product a * b as four 32 x 32 -> 64-bit multiply-adds (each
// one v_mad_u64_u32; no partial sum overflows 64 bits).
__device__ __forceinline__ void mul128(uint64_t a, uint64_t b, uint64_t& lo, uint64_t& hi) {
    const uint32_t a0 = (uint32_t)a, a1 = (uint32_t)(a >> 32);
    const uint32_t b0 = (uint32_t)b, b1 = (uint32_t)(b >> 32);
    const uint64_t p00 = (uint64_t)a0 * b0;
    const uint64_t t1 = (uint64_t)a0 * b1 + (p00 >> 32);
    const uint64_t t2 = (uint64_t)a1 * b0 + (uint32_t)t1;
    hi = (uint64_t)a1 * b1 + ((t1 >> 32) + (t2 >> 32));
    lo = (t2 << 32) | (uint32_t)p00;
}

__device__ __forceinline__ void philox4x64_10(uint64_t (&c)[4], uint64_t k0, uint64_t k1) {
    constexpr uint64_t kM0 = 0xD2E7470EE14C6C93ull, kM1 = 0xCA5A826395121157ull;
    constexpr uint64_t kW0 = 0x9E3779B97F4A7C15ull, kW1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r) {
            k0 += kW0;
            k1 += kW1;
        }
        uint64_t lo0, hi0, lo1, hi1;
        mul128(kM0, c[0], lo0, hi0);
        mul128(kM1, c[2], lo1, hi1);
        const uint64_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
        c[0] = n0;
        c[1] = lo1;
        c[2] = n2;
        c[3] = lo0;
    }
}

// Keep bits of `sites` dropout sites of `words` 32-bit words each: bit b of
// word w of site s is element e = 32 w + b of that site, taken from 32-bit
// word e mod 8 (low half of each 64-bit output first) of Philox4x64-10 at
// counter (e / 8, s, 0, 0) under key (seed, offset); the element is kept when
// that word is at least thr = floor(p 2^32).  One thread per mask word.
__global__ __launch_bounds__(kThreads) void dropout_mask_kernel(uint32_t* __restrict__ mask,
                                                                int64_t words, int64_t total,
                                                                uint32_t thr, uint64_t seed,
                                                                uint64_t offset) {
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i >= total) return;
    const int64_t site = i / words, w = i - site * words;
    uint32_t bits = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        uint64_t c[4] = {(uint64_t)(w * 4 + q), (uint64_t)site, 0ull, 0ull};
        philox4x64_10(c, seed, offset);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            bits |= (uint32_t)((uint32_t)c[j] >= thr) << (8 * q + 2 * j);
            bits |= (uint32_t)((uint32_t)(c[j] >> 32) >= thr) << (8 * q + 2 * j + 1);
        }
    }
    mask[i] = bits;
}

// ------------------------------------------------------------------ LayerNorm
// Four consecutive features per lane (16-byte accesses): a row of D = 64 NV
// features spans G = 16 NV lanes and one wave access covers 64 / G rows.
template <int NV>
struct LnGeo {
    static constexpr int D = 64 * NV;
    static constexpr int G = 16 * NV;     // lanes per row
    static constexpr int RPA = 64 / G;    // rows per wave access
};

// Sum over the G lanes of a row (xor butterfly inside aligned groups of G).
template <int G>
__device__ __forceinline__ float row_sum(float v) {
#pragma unroll
    for (int o = G / 2; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

__device__ __forceinline__ float4 ld4(const float* p) { return *(const float4*)p; }
__device__ __forceinline__ void st4(float* p, float4 v) { *(float4*)p = v; }
__device__ __forceinline__ float el(const float4& v, int i) {
    return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w;
}

// Elements e .. e + 3 of v after dropout (e a multiple of 4: their keep bits
// are bits e % 32 .. + 3 of one word): v * scale where kept, else 0; the
// identity when keep is null (no dropout).
__device__ __forceinline__ float4 drop4(const uint32_t* __restrict__ keep, int64_t e, float4 v,
                                        float scale) {
    if (!keep) return v;
    const uint32_t k = keep[e >> 5] >> (e & 31);
    return float4{(k & 1u) ? v.x * scale : 0.0f, (k & 2u) ? v.y * scale : 0.0f,
                  (k & 4u) ? v.z * scale : 0.0f, (k & 8u) ? v.w * scale : 0.0f};
}

// y = (v - mean) / sqrt(var + eps) * g + b over rows of D = 64 * NV features.
// v = drop(a) + r (r may be null: no residual) and, if s is not null, v is
// stored for the backward (s may be a: in place).  EMB: v is drop(row
// ids[row] of the embedding a), or drop(0) where the id is the padding id
// `pad`; an id outside [0, V) gives NaN.  drop: dropout with the keep bits
// `keep` (null: none) and scale 1 / (1 - p), element index row * D +
// feature.  Each wave normalises kLnRows accesses of RPA rows side by side
// (independent reductions in flight together).
template <int NV, bool EMB>
__global__ __launch_bounds__(kThreads) void ln_fwd_kernel(
    const float* a, const float* r, const int* __restrict__ ids,
    const float* __restrict__ g, const float* __restrict__ b, float* s, float* __restrict__ y,
    float* __restrict__ mu, float* __restrict__ rs, int64_t M, int64_t V, float eps,
    const uint32_t* __restrict__ keep, float scale, int pad) {
    using Geo = LnGeo<NV>;
    constexpr int D = Geo::D, G = Geo::G, RPA = Geo::RPA;
    const int lane = threadIdx.x & (kWave - 1);
    const int sub = lane / G, c = 4 * (lane % G);
    const int64_t row0 = ((int64_t)blockIdx.x * 4 + wave_id()) * (kLnRows * RPA) + sub;
    float4 v[kLnRows];
    float m[kLnRows], rstd[kLnRows];
#pragma unroll
    for (int q = 0; q < kLnRows; ++q) {
        const int64_t rq = row0 + q * RPA;
        const int64_t row = rq < M ? rq : M - 1;  // tail rows recompute row M-1
        const int64_t e = row * D + c;
        if constexpr (EMB) {
            const int64_t id = ids[row];
            const bool ok = id >= 0 && id < V;
            const bool padded = pad >= 0 && id == pad;
            const float bad = ok ? 0.0f : __builtin_nanf("");
            float4 t = padded ? float4{0.0f, 0.0f, 0.0f, 0.0f} : ld4(a + (ok ? id : 0) * D + c);
            t = drop4(keep, e, t, scale);
            v[q] = float4{t.x + bad, t.y + bad, t.z + bad, t.w + bad};
        } else {
            float4 t = drop4(keep, e, ld4(a + e), scale);
            if (r) {
                const float4 u = ld4(r + e);
                t = float4{t.x + u.x, t.y + u.y, t.z + u.z, t.w + u.w};
            }
            v[q] = t;
        }
    }
#pragma unroll
    for (int q = 0; q < kLnRows; ++q)
        m[q] = row_sum<G>((v[q].x + v[q].y) + (v[q].z + v[q].w)) * (1.0f / D);
#pragma unroll
    for (int q = 0; q < kLnRows; ++q) {
        const float dx0 = v[q].x - m[q], dx1 = v[q].y - m[q], dx2 = v[q].z - m[q],
                    dx3 = v[q].w - m[q];
        const float var = (dx0 * dx0 + dx1 * dx1) + (dx2 * dx2 + dx3 * dx3);
        rstd[q] = 1.0f / sqrtf(row_sum<G>(var) * (1.0f / D) + eps);
    }
    const float4 gc = ld4(g + c), bc = ld4(b + c);
#pragma unroll
    for (int q = 0; q < kLnRows; ++q) {
        const int64_t row = row0 + q * RPA;
        if (row >= M) break;
        const int64_t e = row * D + c;
        if (s) st4(s + e, v[q]);
        st4(y + e, float4{(v[q].x - m[q]) * rstd[q] * gc.x + bc.x,
                          (v[q].y - m[q]) * rstd[q] * gc.y + bc.y,
                          (v[q].z - m[q]) * rstd[q] * gc.z + bc.z,
                          (v[q].w - m[q]) * rstd[q] * gc.w + bc.w});
        if (c == 0) {
            mu[row] = m[q];
            rs[row] = rstd[q];
        }
    }
}

// LayerNorm backward: dv = rstd (gd - mean(gd) - xh mean(gd xh)), gd = dy g,
// xh = (v - mean) rstd with v from s (or, EMB, recomputed from the embedding
// rows by id, the padding id and the keep bits as in the forward).  Non-EMB:
// dx = dv (the residual's gradient) and, if dxm is not null, dxm = dv through
// the dropout (the sub-layer output's gradient).  EMB: dx = dv through the
// dropout, 0 at padded positions (the gradient of the looked-up rows).
// DROP: keep bits given (and, non-EMB, dxm with them); without, neither.  The
// workgroup handles rows [blk * kLnBwdRows, + kLnBwdRows) in wave accesses of
// RPA rows (wave w takes accesses w, w + 4, ...); each lane sums dy xh and dy
// of its four features over its rows in order, then the RPA row slots of a
// wave and the four waves are added in a fixed order into pg[blk], pb[blk]
// (summed over workgroups later).
template <int NV, bool EMB, bool DROP>
__global__ __launch_bounds__(kThreads) void ln_bwd_kernel(
    const float* __restrict__ dy, const float* __restrict__ s, const int* __restrict__ ids,
    const float* __restrict__ mu, const float* __restrict__ rs, const float* __restrict__ g,
    float* __restrict__ dx, float* __restrict__ pg, float* __restrict__ pb, int64_t M,
    int64_t V, const uint32_t* __restrict__ keep, float scale, int pad,
    float* __restrict__ dxm) {
    using Geo = LnGeo<NV>;
    constexpr int D = Geo::D, G = Geo::G, RPA = Geo::RPA;
    __shared__ float4 red[4][2][D / 4];
    const int lane = threadIdx.x & (kWave - 1), w = wave_id();
    const int sub = lane / G, c = 4 * (lane % G);
    const int64_t r0 = (int64_t)blockIdx.x * kLnBwdRows;
    const int64_t r1 = r0 + kLnBwdRows < M ? r0 + kLnBwdRows : M;
    float4 ag{0.0f, 0.0f, 0.0f, 0.0f}, ab{0.0f, 0.0f, 0.0f, 0.0f};
    const float4 gc = ld4(g + c);
    // A row's inputs (the normalised value's source, dy, the row statistics
    // and the keep bits of the lane's four elements), all read before the
    // stores that use them: vector memory operations complete in issue
    // order, so a read issued after a store is waited for together with it.
    struct RowRaw {
        float4 v, d;
        float m, rstd;
        uint32_t kw;
        bool padded;
    };
    struct RowIn {
        float4 xh, d, gd;
        float s1, s2, rstd;
        uint32_t kw;
        bool padded;
    };
    auto drop_bits = [&](uint32_t k, float4 v) -> float4 {
        if constexpr (!DROP) return v;
        return float4{(k & 1u) ? v.x * scale : 0.0f, (k & 2u) ? v.y * scale : 0.0f,
                      (k & 4u) ? v.z * scale : 0.0f, (k & 8u) ? v.w * scale : 0.0f};
    };
    auto row_load = [&](int64_t row, RowRaw& r) {
        const int64_t e = row * D + c;
        if constexpr (EMB) {
            const int64_t id = ids[row];
            r.padded = pad >= 0 && id == pad;
            r.v = r.padded ? float4{0.0f, 0.0f, 0.0f, 0.0f}
                           : ld4(s + (id >= 0 && id < V ? id : 0) * D + c);
        } else {
            r.padded = false;
            r.v = ld4(s + e);
        }
        if constexpr (DROP)
            r.kw = keep[e >> 5] >> (e & 31);
        else
            r.kw = 0xFu;
        r.m = mu[row];
        r.rstd = rs[row];
        r.d = ld4(dy + e);
    };
    auto row_grad = [&](const RowRaw& r, RowIn& o) {
        const float4 v = EMB ? drop_bits(r.kw, r.v) : r.v;
        const float m = r.m, rstd = r.rstd;
        o.xh = float4{(v.x - m) * rstd, (v.y - m) * rstd, (v.z - m) * rstd, (v.w - m) * rstd};
        o.d = r.d;
        o.gd = float4{o.d.x * gc.x, o.d.y * gc.y, o.d.z * gc.z, o.d.w * gc.w};
        o.s1 = (o.gd.x + o.gd.y) + (o.gd.z + o.gd.w);
        o.s2 = (o.gd.x * o.xh.x + o.gd.y * o.xh.y) + (o.gd.z * o.xh.z + o.gd.w * o.xh.w);
        o.rstd = rstd;
        o.kw = r.kw;
        o.padded = r.padded;
    };
    auto row_out = [&](int64_t row, const RowIn& o, float m1, float m2) {
        const float rstd = o.rstd;
        const int64_t e = row * D + c;
        const float4 dv{rstd * (o.gd.x - m1 - o.xh.x * m2), rstd * (o.gd.y - m1 - o.xh.y * m2),
                        rstd * (o.gd.z - m1 - o.xh.z * m2), rstd * (o.gd.w - m1 - o.xh.w * m2)};
        if constexpr (EMB) {
            st4(dx + e, o.padded ? float4{0.0f, 0.0f, 0.0f, 0.0f} : drop_bits(o.kw, dv));
        } else {
            st4(dx + e, dv);
            if constexpr (DROP) st4(dxm + e, drop_bits(o.kw, dv));
        }
        ag = float4{fmaf(o.d.x, o.xh.x, ag.x), fmaf(o.d.y, o.xh.y, ag.y),
                    fmaf(o.d.z, o.xh.z, ag.z), fmaf(o.d.w, o.xh.w, ag.w)};
        ab = float4{ab.x + o.d.x, ab.y + o.d.y, ab.z + o.d.z, ab.w + o.d.w};
    };
    // Accesses w, w + 4, ... of the block, two at a time so that their loads
    // and reductions overlap, the next pair's inputs read before this pair's
    // stores; rows past r1 are skipped (all RPA rows of an access are in
    // range or not, per lane).
    int64_t row = r0 + (int64_t)w * RPA + sub;
    constexpr int64_t kStep = 4 * RPA;
    RowRaw xa, xb;
    if (row + kStep < r1) {
        row_load(row, xa);
        row_load(row + kStep, xb);
    }
    for (; row + kStep < r1; row += 2 * kStep) {
        RowIn ia, ib;
        row_grad(xa, ia);
        row_grad(xb, ib);
        // (rows clamped to r1 - 1 past the block, read but unused: the loop
        // then issues the same memory operations every pass, so the
        // compiler's wait counts stay exact)
        const int64_t nr = row + 2 * kStep;
        row_load(nr < r1 ? nr : r1 - 1, xa);
        row_load(nr + kStep < r1 ? nr + kStep : r1 - 1, xb);
        const float m1a = row_sum<G>(ia.s1) * (1.0f / D), m2a = row_sum<G>(ia.s2) * (1.0f / D);
        const float m1b = row_sum<G>(ib.s1) * (1.0f / D), m2b = row_sum<G>(ib.s2) * (1.0f / D);
        row_out(row, ia, m1a, m2a);
        row_out(row + kStep, ib, m1b, m2b);
    }
    {
        // The last access: rows before r1 only.  The sums are taken by every
        // lane of the wave (the shuffles need all of them); out-of-range rows
        // read row r1 - 1 and store nothing.
        const bool in = row < r1;
        RowRaw xr;
        row_load(in ? row : r1 - 1, xr);
        RowIn ia;
        row_grad(xr, ia);
        const float m1a = row_sum<G>(ia.s1) * (1.0f / D), m2a = row_sum<G>(ia.s2) * (1.0f / D);
        if (in) row_out(row, ia, m1a, m2a);
    }
    // The RPA row slots of the wave (lanes G apart), then the four waves.
#pragma unroll
    for (int o = G; o < kWave; o <<= 1) {
        ag = float4{ag.x + __shfl_xor(ag.x, o), ag.y + __shfl_xor(ag.y, o),
                    ag.z + __shfl_xor(ag.z, o), ag.w + __shfl_xor(ag.w, o)};
        ab = float4{ab.x + __shfl_xor(ab.x, o), ab.y + __shfl_xor(ab.y, o),
                    ab.z + __shfl_xor(ab.z, o), ab.w + __shfl_xor(ab.w, o)};
    }
    if (sub == 0) {
        red[w][0][c / 4] = ag;
        red[w][1][c / 4] = ab;
    }
    __syncthreads();
    if (w == 0 && sub == 0) {
        float4 tg = red[0][0][c / 4], tb = red[0][1][c / 4];
#pragma unroll
        for (int q = 1; q < 4; ++q) {
            const float4 ug = red[q][0][c / 4], ub = red[q][1][c / 4];
            tg = float4{tg.x + ug.x, tg.y + ug.y, tg.z + ug.z, tg.w + ug.w};
            tb = float4{tb.x + ub.x, tb.y + ub.y, tb.z + ub.z, tb.w + ub.w};
        }
        st4(pg + blockIdx.x * D + c, tg);
        st4(pb + blockIdx.x * D + c, tb);
    }
}

// ------------------------------------------------------------------ elementwise
// C[m][n] = bias[n] (the GEMM then accumulates onto it).
__global__ __launch_bounds__(kThreads) void bias_rows_kernel(const float* __restrict__ bias,
                                                             float* __restrict__ C, int64_t M,
                                                             int64_t N) {
    const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (e * 4 >= M * N) return;
    const int64_t n = (e * 4) % N;  // N % 4 == 0
    *(float4*)(C + e * 4) = *(const float4*)(bias + n);
}

__global__ __launch_bounds__(kThreads) void silu_fwd_kernel(const float* __restrict__ A,
                                                            float* __restrict__ P, int64_t n) {
    const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (e * 4 >= n) return;
    float4 a = *(const float4*)(A + e * 4);
    a.x *= sigmoid(a.x);
    a.y *= sigmoid(a.y);
    a.z *= sigmoid(a.z);
    a.w *= sigmoid(a.w);
    *(float4*)(P + e * 4) = a;
}

// dA = dP SiLU'(A), SiLU'(v) = s (1 + v (1 - s)), in place over dP.
__global__ __launch_bounds__(kThreads) void silu_bwd_kernel(float* __restrict__ dP,
                                                            const float* __restrict__ A,
                                                            int64_t n) {
    const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (e * 4 >= n) return;
    const float4 a = *(const float4*)(A + e * 4);
    float4 d = *(const float4*)(dP + e * 4);
    const float av[4] = {a.x, a.y, a.z, a.w};
    float dv[4] = {d.x, d.y, d.z, d.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float sg = sigmoid(av[i]);
        dv[i] *= sg * fmaf(av[i], 1.0f - sg, 1.0f);
    }
    *(float4*)(dP + e * 4) = make_float4(dv[0], dv[1], dv[2], dv[3]);
}

// ------------------------------------------------------------------ prediction and loss
// Block sum / max over 256 threads in a fixed tree order.
template <bool MAX>
__device__ __forceinline__ float block_reduce(float v, float* sh) {
    sh[threadIdx.x] = v;
    __syncthreads();
    for (int o = kThreads / 2; o > 0; o >>= 1) {
        if ((int)threadIdx.x < o)
            sh[threadIdx.x] = MAX ? fmaxf(sh[threadIdx.x], sh[threadIdx.x + o])
                                  : sh[threadIdx.x] + sh[threadIdx.x + o];
        __syncthreads();
    }
    const float r = sh[0];
    __syncthreads();
    return r;
}

// Row b of the logits: loss_b = logsumexp - logit[target], and
// dlogits = (softmax - onehot(target)) / B.  A target outside [0, V) gives NaN.
__global__ __launch_bounds__(kThreads) void ce_kernel(const float* __restrict__ logits,
                                                      const int* __restrict__ targets, int64_t B,
                                                      int64_t V, float* __restrict__ dlogits,
                                                      float* __restrict__ lossb) {
    __shared__ float sh[kThreads];
    const int64_t b = blockIdx.x;
    const float* l = logits + b * V;
    float mx = -__builtin_huge_valf();
    for (int64_t v = threadIdx.x; v < V; v += kThreads) mx = fmaxf(mx, l[v]);
    mx = block_reduce<true>(mx, sh);
    float se = 0.0f;
    for (int64_t v = threadIdx.x; v < V; v += kThreads) se += expf(l[v] - mx);
    se = block_reduce<false>(se, sh);
    const int64_t t = targets[b];
    const bool ok = t >= 0 && t < V;
    const float inv = 1.0f / se, scale = 1.0f / (float)B;
    for (int64_t v = threadIdx.x; v < V; v += kThreads)
        dlogits[b * V + v] = (expf(l[v] - mx) * inv - (v == t ? 1.0f : 0.0f)) * scale;
    if (threadIdx.x == 0) lossb[b] = ok ? logf(se) + mx - l[t] : __builtin_nanf("");
}

// loss = sum_b loss_b / B in double, in a fixed order: thread t adds rows
// t, t + 256, ... in turn, then the 256 partials are added in a fixed tree
// (one workgroup of kThreads).
__global__ __launch_bounds__(kThreads) void loss_final_kernel(const float* __restrict__ lossb,
                                                              int64_t B,
                                                              float* __restrict__ loss) {
    __shared__ double sh[kThreads];
    double acc = 0.0;
    for (int64_t b = threadIdx.x; b < B; b += kThreads) acc += (double)lossb[b];
    sh[threadIdx.x] = acc;
    __syncthreads();
    for (int o = kThreads / 2; o > 0; o >>= 1) {
        if ((int)threadIdx.x < o) sh[threadIdx.x] += sh[threadIdx.x + o];
        __syncthreads();
    }
    if (threadIdx.x == 0) *loss = (float)(sh[0] / (double)B);
}

// ------------------------------------------------------------------ embedding gradient
__global__ void iota_kernel(int* __restrict__ p, int64_t n) {
    const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (e < n) p[e] = (int)e;
}

__device__ __forceinline__ int64_t lower_bound_u32(const unsigned* a, int64_t n, unsigned key) {
    int64_t lo = 0, hi = n;
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (a[mid] < key) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

// The input side of dE: for each item v, the rows of dx at the positions
// holding v, summed in position order (ids sorted stably with their
// positions).  Popular items hold many positions, so the work is cut into
// pieces of kPiece sorted positions: item v has ceil(n_v / kPiece) pieces
// starting at poff[v] (an exclusive scan); one wave sums each piece, then one
// wave per item adds its pieces in order.
constexpr int64_t kPiece = 256;

__global__ __launch_bounds__(kThreads) void emb_count_kernel(const unsigned* __restrict__ ids_sorted,
                                                             int64_t M, int64_t V,
                                                             int64_t* __restrict__ lo,
                                                             int64_t* __restrict__ hi,
                                                             int64_t* __restrict__ npiece) {
    const int64_t v = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (v >= V) return;
    const int64_t a = lower_bound_u32(ids_sorted, M, (unsigned)v);
    const int64_t b = lower_bound_u32(ids_sorted, M, (unsigned)v + 1u);
    lo[v] = a;
    hi[v] = b;
    npiece[v] = (b - a + kPiece - 1) / kPiece;
}

// out[i] = sum of in[0 .. i) for i <= n (one workgroup of 1024 threads).
__global__ __launch_bounds__(1024) void exclusive_scan_kernel(const int64_t* __restrict__ in,
                                                              int64_t* __restrict__ out,
                                                              int64_t n) {
    __shared__ int64_t buf[2][1024];
    const int t = threadIdx.x;
    int64_t carry = 0;
    for (int64_t base = 0; base < n; base += 1024) {
        const int64_t x = base + t < n ? in[base + t] : 0;
        int cur = 0;
        buf[cur][t] = x;
        __syncthreads();
        for (int o = 1; o < 1024; o <<= 1) {
            const int64_t v = buf[cur][t] + (t >= o ? buf[cur][t - o] : 0);
            buf[cur ^ 1][t] = v;
            cur ^= 1;
            __syncthreads();
        }
        if (base + t < n) out[base + t] = carry + buf[cur][t] - x;
        carry += buf[cur][1023];
        __syncthreads();
    }
    if (t == 0) out[n] = carry;
}

template <int NV>
__global__ __launch_bounds__(kThreads) void emb_piece_kernel(
    const int* __restrict__ pos_sorted, const float* __restrict__ dx,
    const int64_t* __restrict__ lo, const int64_t* __restrict__ hi,
    const int64_t* __restrict__ poff, float* __restrict__ part, int64_t V, int64_t max_pieces) {
    constexpr int D = 64 * NV;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t p = (int64_t)blockIdx.x * 4 + wave_id();
    if (p >= max_pieces || p >= poff[V]) return;
    // the item whose pieces contain p: the last v with poff[v] <= p
    int64_t a = 0, b = V;
    while (b - a > 1) {
        const int64_t mid = (a + b) >> 1;
        if (poff[mid] <= p) a = mid;
        else b = mid;
    }
    const int64_t start = lo[a] + (p - poff[a]) * kPiece;
    const int64_t end = start + kPiece < hi[a] ? start + kPiece : hi[a];
    float acc[NV];
#pragma unroll
    for (int j = 0; j < NV; ++j) acc[j] = 0.0f;
    // kBatch positions' rows loaded together, then added in position order
    constexpr int kBatch = 8;
    int64_t i = start;
    for (; i + kBatch <= end; i += kBatch) {
        int64_t r[kBatch];
        float v[kBatch][NV];
#pragma unroll
        for (int q = 0; q < kBatch; ++q) r[q] = pos_sorted[i + q];
#pragma unroll
        for (int q = 0; q < kBatch; ++q)
#pragma unroll
            for (int j = 0; j < NV; ++j) v[q][j] = dx[r[q] * D + lane + 64 * j];
#pragma unroll
        for (int q = 0; q < kBatch; ++q)
#pragma unroll
            for (int j = 0; j < NV; ++j) acc[j] += v[q][j];
    }
    for (; i < end; ++i) {
        const int64_t r = pos_sorted[i];
#pragma unroll
        for (int j = 0; j < NV; ++j) acc[j] += dx[r * D + lane + 64 * j];
    }
#pragma unroll
    for (int j = 0; j < NV; ++j) part[p * D + lane + 64 * j] = acc[j];
}

template <int NV>
__global__ __launch_bounds__(kThreads) void emb_item_kernel(const int64_t* __restrict__ poff,
                                                            const float* __restrict__ part,
                                                            float* __restrict__ dE, int64_t V) {
    constexpr int D = 64 * NV;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t v = (int64_t)blockIdx.x * 4 + wave_id();
    if (v >= V || poff[v] == poff[v + 1]) return;
    float acc[NV];
#pragma unroll
    for (int j = 0; j < NV; ++j) acc[j] = 0.0f;
    // kBatch pieces loaded together, then added in piece order
    constexpr int kBatch = 8;
    const int64_t p1 = poff[v + 1];
    int64_t p = poff[v];
    for (; p + kBatch <= p1; p += kBatch) {
        float x[kBatch][NV];
#pragma unroll
        for (int q = 0; q < kBatch; ++q)
#pragma unroll
            for (int j = 0; j < NV; ++j) x[q][j] = part[(p + q) * D + lane + 64 * j];
#pragma unroll
        for (int q = 0; q < kBatch; ++q)
#pragma unroll
            for (int j = 0; j < NV; ++j) acc[j] += x[q][j];
    }
    for (; p < p1; ++p)
#pragma unroll
        for (int j = 0; j < NV; ++j) acc[j] += part[p * D + lane + 64 * j];
#pragma unroll
    for (int j = 0; j < NV; ++j) dE[v * D + lane + 64 * j] += acc[j];
}

// ------------------------------------------------------------------ Adam
// Kingma and Ba, Algorithm 1: m = b1 m + (1 - b1) g, v = b2 v + (1 - b2) g^2,
// p -= lr (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps).
__global__ __launch_bounds__(kThreads) void adam_kernel(float* __restrict__ p,
                                                        const float* __restrict__ g,
                                                        float* __restrict__ m1,
                                                        float* __restrict__ m2, int64_t n,
                                                        float lr, float b1, float b2, float eps,
                                                        float c1, float c2) {
    const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (e >= n) return;
    const float gv = g[e];
    const float a = b1 * m1[e] + (1.0f - b1) * gv;
    const float b = b2 * m2[e] + (1.0f - b2) * gv * gv;
    m1[e] = a;
    m2[e] = b;
    p[e] -= lr * (a / c1) / (sqrtf(b / c2) + eps);
}

unsigned blocks_for(int64_t n, int64_t per = kThreads) { return (unsigned)((n + per - 1) / per); }

}  // namespace

// ------------------------------------------------------------------ parameter layout
int64_t layer_tensor_size(const Dims& d, int k) {
    const int64_t D = d.D, ED = d.E * d.D, F = 4 * d.D;
    switch (k) {
        case kWx: case kWz: return ED * D;
        case kConvW: return ED * d.K;
        case kWr: case kWi: return ED * ED;
        case kWo: return D * ED;
        case kW1: return F * D;
        case kb1: return F;
        case kW2: return D * F;
        case kbo: case kLn1g: case kLn1b: case kb2: case kLn2g: case kLn2b: return D;
        default: return ED;  // bx, bz, conv_b, br, bi, lambda
    }
}

int64_t tensor_count(const Dims& d) { return 3 + kLayerTensors * d.layers; }

// Offsets (floats) of every tensor in order; returns the total (a multiple of 64).
int64_t param_offsets(const Dims& d, int64_t* off) {
    int64_t at = 0, i = 0;
    auto put = [&](int64_t size) {
        if (off) off[i] = at;
        ++i;
        at += (size + 63) / 64 * 64;
    };
    put(d.V * d.D);
    put(d.D);
    put(d.D);
    for (int64_t l = 0; l < d.layers; ++l)
        for (int k = 0; k < kLayerTensors; ++k) put(layer_tensor_size(d, k));
    return at;
}

// ------------------------------------------------------------------ workspace
struct Layout {
    size_t H, Hx, Hz, hb, y, s1, H1, A, P, s2, stats, emb_stats, logits, dlogits, lossb;
    size_t X, Y, Z, dP, dY, dHx, dHz, lnp, dwp, wt, colsum, emb_lo, emb_hi, emb_np, emb_poff,
        emb_part, mask;
    size_t ids_s, pos, pos_s, sort_tmp, gated, total;
    size_t sort_bytes, gated_bytes;
};

constexpr int64_t kDwChunk = 4096;  // rows per partial of a weight gradient

// Dropout sites (the embedding, then two per layer) and 32-bit keep words per
// site (B T D is a multiple of 64).
int64_t mask_sites(const Dims& d) { return 1 + 2 * d.layers; }
int64_t mask_words(const Dims& d) { return d.B * d.T * d.D / 32; }

Layout layout(const Dims& d) {
    const int64_t M = d.B * d.T, D = d.D, ED = d.E * d.D, F = 4 * d.D, L = d.layers;
    const size_t f = sizeof(float);
    Layout w{};
    size_t at = 0;
    auto take = [&](size_t bytes) {
        const size_t o = at;
        at += align_up(bytes);
        return o;
    };
    w.H = take((size_t)((L + 1) * M * D) * f);  // layer inputs / outputs
    w.Hx = take((size_t)(L * M * ED) * f);
    w.Hz = take((size_t)(L * M * ED) * f);
    w.hb = take((size_t)(L * M * ED) * f);      // BD-LRU outputs
    w.y = take((size_t)(L * M * ED) * f);
    w.s1 = take((size_t)(L * M * D) * f);
    w.H1 = take((size_t)(L * M * D) * f);
    w.A = take((size_t)(L * M * F) * f);
    w.P = take((size_t)(L * M * F) * f);
    w.s2 = take((size_t)(L * M * D) * f);
    w.stats = take((size_t)(L * 4 * M) * f);    // mean and 1/std of both LayerNorms
    w.emb_stats = take((size_t)(2 * M) * f);
    w.logits = take((size_t)(d.B * d.V) * f);
    w.dlogits = take((size_t)(d.B * d.V) * f);
    w.lossb = take((size_t)d.B * f);
    w.X = take((size_t)(M * D) * f);
    w.Y = take((size_t)(M * D) * f);
    w.Z = take((size_t)(M * D) * f);            // a sub-layer output's gradient (dropout)
    w.dP = take((size_t)(M * F) * f);
    w.dY = take((size_t)(M * ED) * f);
    w.dHx = take((size_t)(M * ED) * f);
    w.dHz = take((size_t)(M * ED) * f);
    const int64_t lnblk = (M + kLnBwdRows - 1) / kLnBwdRows;
    w.lnp = take((size_t)(2 * lnblk * D) * f);
    // weight gradients: one partial per chunk of kDwChunk rows, summed after
    const int64_t NK = 4 * D * D > ED * D ? 4 * D * D : ED * D;
    const int64_t slices = M / kDwChunk + 1;
    // (or, on the matrix-core path, one partial per split of the rows, and
    // the bias gradient's partials after them)
    const int64_t wshape[4][2] = {{D, F}, {F, D}, {D, ED}, {ED, D}};
    size_t dwp = (size_t)(slices * NK) * f;
    for (const auto& nk : wshape)
        if (wgrad_workspace(M, nk[0], nk[1]) > dwp) dwp = wgrad_workspace(M, nk[0], nk[1]);
    w.dwp = take(dwp);
    w.wt = take((size_t)NK * f);  // a transposed weight (data gradients)
    // column sums: bias gradients (widths D, 4D, E*D), LayerNorm partials, the
    // weight-gradient slices or splits
    size_t cs = colsum_workspace(M, F > ED ? F : ED);
    if (colsum_workspace(lnblk, D) > cs) cs = colsum_workspace(lnblk, D);
    if (colsum_workspace(slices, NK) > cs) cs = colsum_workspace(slices, NK);
    for (const auto& nk : wshape) {
        const int64_t sp = wgrad_splits(M, nk[0], nk[1]);
        if (colsum_workspace(sp, nk[0] * nk[1]) > cs) cs = colsum_workspace(sp, nk[0] * nk[1]);
    }
    w.colsum = take(cs);
    const int64_t max_pieces = (M + kPiece - 1) / kPiece + d.V;
    w.emb_lo = take((size_t)d.V * sizeof(int64_t));
    w.emb_hi = take((size_t)d.V * sizeof(int64_t));
    w.emb_np = take((size_t)(d.V + 1) * sizeof(int64_t));
    w.emb_poff = take((size_t)(d.V + 1) * sizeof(int64_t));
    w.emb_part = take((size_t)(max_pieces * D) * f);
    w.mask = take((size_t)(mask_sites(d) * mask_words(d)) * sizeof(uint32_t));
    w.ids_s = take((size_t)M * sizeof(unsigned));
    w.pos = take((size_t)M * sizeof(int));
    w.pos_s = take((size_t)M * sizeof(int));
    size_t sb = 0;
    hipcub::DeviceRadixSort::SortPairs(nullptr, sb, (const unsigned*)nullptr, (unsigned*)nullptr,
                                       (const int*)nullptr, (int*)nullptr, (int)M, 0, 32);
    w.sort_bytes = sb;
    w.sort_tmp = take(sb);
    const size_t gf = recblr_workspace_size(RECBLR_OP_GATED_FORWARD, d.B, d.T, ED, RECBLR_F32);
    const size_t gb = recblr_workspace_size(RECBLR_OP_GATED_BACKWARD, d.B, d.T, ED, RECBLR_F32);
    w.gated_bytes = gf > gb ? gf : gb;
    w.gated = take(w.gated_bytes);
    w.total = at;
    return w;
}

size_t workspace_size(const Dims& d) { return layout(d).total; }

// ------------------------------------------------------------------ runner
namespace {

struct Ctx {
    rocblas_handle blas;
    hipStream_t stream;
    char* ws;
    const Layout& w;
    bool ok = true;
};

// Row-major Y[M][N] (+)= X[M][K] W[N][K]^T: column-major Y^T = W X^T.
bool gemm_xwT(Ctx& c, const float* X, int64_t ldx, const float* W, float* Y, int64_t ldy,
              int64_t M, int64_t N, int64_t K, float beta) {
    const float one = 1.0f;
    return rocblas_sgemm(c.blas, rocblas_operation_transpose, rocblas_operation_none, (int)N,
                         (int)M, (int)K, &one, W, (int)K, X, (int)ldx, &beta, Y,
                         (int)ldy) == rocblas_status_success;
}
// Row-major dX[M][K] (+)= dY[M][N] W[N][K]: column-major dX^T = W^T dY^T.
bool gemm_dyW(Ctx& c, const float* dY, int64_t lddy, const float* W, float* dX, int64_t lddx,
              int64_t M, int64_t N, int64_t K, float beta) {
    const float one = 1.0f;
    return rocblas_sgemm(c.blas, rocblas_operation_none, rocblas_operation_none, (int)K, (int)M,
                         (int)N, &one, W, (int)K, dY, (int)lddy, &beta, dX,
                         (int)lddx) == rocblas_status_success;
}
// Row-major dW[N][K] = dY[M][N]^T X[M][K]: column-major dW^T = X^T dY.
bool gemm_dyTx(Ctx& c, const float* X, int64_t ldx, const float* dY, int64_t lddy, float* dW,
               int64_t M, int64_t N, int64_t K) {
    const float one = 1.0f, zero = 0.0f;
    return rocblas_sgemm(c.blas, rocblas_operation_none, rocblas_operation_transpose, (int)K,
                         (int)N, (int)M, &one, X, (int)ldx, dY, (int)lddy, &zero, dW,
                         (int)K) == rocblas_status_success;
}

// dW[N][K] = dY^T X over M rows: a GEMM per chunk of kDwChunk rows (one
// strided-batched call), then the chunk partials summed in order (double).
// A single GEMM over all rows would reduce along 409,600 rows inside the
// library, which its kernels do slowly.
bool weight_grad(Ctx& c, const float* X, int64_t ldx, const float* dY, int64_t lddy, float* dW,
                 int64_t M, int64_t N, int64_t K) {
    const int64_t nb = M / kDwChunk, rem = M - nb * kDwChunk;
    if (nb < 2) return gemm_dyTx(c, X, ldx, dY, lddy, dW, M, N, K);
    float* part = (float*)(c.ws + c.w.dwp);
    const float one = 1.0f, zero = 0.0f;
    if (rocblas_sgemm_strided_batched(c.blas, rocblas_operation_none, rocblas_operation_transpose,
                                      (int)K, (int)N, (int)kDwChunk, &one, X, (int)ldx,
                                      kDwChunk * ldx, dY, (int)lddy, kDwChunk * lddy, &zero, part,
                                      (int)K, K * N, (int)nb) != rocblas_status_success)
        return false;
    int64_t slices = nb;
    if (rem > 0) {
        if (!gemm_dyTx(c, X + nb * kDwChunk * ldx, ldx, dY + nb * kDwChunk * lddy, lddy,
                       part + nb * K * N, rem, N, K))
            return false;
        ++slices;
    }
    return launch_colsum(part, slices, N * K, dW, c.ws + c.w.colsum, c.stream) == hipSuccess;
}

// Y[M][N] = X[M][K] W[N][K]^T + b; act, if given, gets SiLU(Y).  On the
// library's fp32 matrix-core tiles with the bias and the SiLU in the
// epilogue when the operands allow (always, for the model's shapes and
// workspace), else bias rows, a library GEMM and a SiLU pass.
bool linear_fwd(Ctx& c, const float* X, const float* W, const float* b, float* Y, int64_t M,
                int64_t N, int64_t K, float* act = nullptr) {
    if (wgrad_fast_ok({X, W, b, Y, act}, M, N, K))
        return launch_linear_fwd32(X, W, b, Y, act, M, N, K, c.stream) == hipSuccess;
    hipLaunchKernelGGL(bias_rows_kernel, dim3(blocks_for(M * N / 4)), dim3(kThreads), 0, c.stream,
                       b, Y, M, N);
    if (hipGetLastError() != hipSuccess) return false;
    if (!gemm_xwT(c, X, K, W, Y, N, M, N, K, 1.0f)) return false;
    if (!act) return true;
    hipLaunchKernelGGL(silu_fwd_kernel, dim3(blocks_for(M * N / 4)), dim3(kThreads), 0, c.stream,
                       Y, act, M * N);
    return hipGetLastError() == hipSuccess;
}

// Data gradient of Y = X W^T: dX[M][K] = dY[M][N] W[N][K] (kStore), dX += it
// (kAccumulate), or dX = it * SiLU'(A) with A[M][K] the SiLU's input
// (kSiluGrad); same choice of path as linear_fwd.
bool linear_dgrad(Ctx& c, const float* dY, const float* W, float* dX, int64_t M, int64_t N,
                  int64_t K, LinearMode mode, const float* A = nullptr) {
    float* wt = (float*)(c.ws + c.w.wt);
    if (wgrad_fast_ok({dY, W, dX, A, wt}, M, N, K))
        return launch_linear_dgrad32(dY, W, dX, mode, A, M, N, K, wt, c.stream) == hipSuccess;
    if (!gemm_dyW(c, dY, N, W, dX, K, M, N, K, mode == LinearMode::kAccumulate ? 1.0f : 0.0f))
        return false;
    if (mode != LinearMode::kSiluGrad) return true;
    hipLaunchKernelGGL(silu_bwd_kernel, dim3(blocks_for(M * K / 4)), dim3(kThreads), 0, c.stream,
                       dX, A, M * K);
    return hipGetLastError() == hipSuccess;
}

// db[n] = sum_m dY[m][n] in a fixed order (double).
bool bias_grad(Ctx& c, const float* dY, int64_t M, int64_t N, float* db) {
    return launch_colsum(dY, M, N, db, c.ws + c.w.colsum, c.stream) == hipSuccess;
}

// Weight and bias gradients of Y = X W^T + b: dW[N][K] = dY^T X and db =
// column sums of dY, both in a fixed order; on the matrix-core tiles when the
// operands allow (always, for the model's shapes and workspace), else a
// library GEMM per chunk of rows and column sums.
bool linear_wgrad(Ctx& c, const float* X, const float* dY, float* dW, float* db, int64_t M,
                  int64_t N, int64_t K) {
    if (wgrad_fast_ok({X, dY, dW, db}, M, N, K))
        return launch_wgrad(dY, X, dW, db, M, N, K, c.ws + c.w.dwp, c.ws + c.w.colsum,
                            c.stream) == hipSuccess;
    return bias_grad(c, dY, M, N, db) && weight_grad(c, X, K, dY, N, dW, M, N, K);
}

// Dropout of one site: its keep bits (null: no dropout), 1 / (1 - p), and the
// padding id (embedding site only; -1: none).
struct Drop {
    const uint32_t* keep = nullptr;
    float scale = 1.0f;
    int pad = -1;
};

template <int NV>
bool ln_fwd(Ctx& c, const float* a, const float* r, const int* ids, const float* g,
            const float* b, float* s, float* y, float* mu, float* rs, int64_t M, int64_t V,
            float eps, Drop dr) {
    const dim3 grid(blocks_for(M, 4 * kLnRows * LnGeo<NV>::RPA));
    if (ids)
        hipLaunchKernelGGL((ln_fwd_kernel<NV, true>), grid, dim3(kThreads), 0, c.stream, a, r,
                           ids, g, b, s, y, mu, rs, M, V, eps, dr.keep, dr.scale, dr.pad);
    else
        hipLaunchKernelGGL((ln_fwd_kernel<NV, false>), grid, dim3(kThreads), 0, c.stream, a, r,
                           ids, g, b, s, y, mu, rs, M, V, eps, dr.keep, dr.scale, dr.pad);
    return hipGetLastError() == hipSuccess;
}

// LayerNorm backward; gamma / beta gradients into dg, db; dxm (non-embedding,
// may be null) the gradient of the dropped-out sub-layer output.
template <int NV>
bool ln_bwd(Ctx& c, const float* dy, const float* s, const int* ids, const float* mu,
            const float* rs, const float* g, float* dx, float* dg, float* db, int64_t M,
            int64_t V, Drop dr, float* dxm = nullptr) {
    constexpr int D = 64 * NV;
    const int64_t nblk = (M + kLnBwdRows - 1) / kLnBwdRows;
    float* pg = (float*)(c.ws + c.w.lnp);
    float* pb = pg + nblk * D;
    // The kernel reads the keep bits and writes dxm together (non-EMB).
    const bool drop = dr.keep != nullptr;
    if (!ids && drop != (dxm != nullptr)) return false;
    auto run = [&](auto emb, auto dp) {
        hipLaunchKernelGGL((ln_bwd_kernel<NV, decltype(emb)::value, decltype(dp)::value>),
                           dim3((unsigned)nblk), dim3(kThreads), 0, c.stream, dy, s, ids, mu, rs,
                           g, dx, pg, pb, M, V, dr.keep, dr.scale, dr.pad, dxm);
    };
    using T_ = std::true_type;
    using F_ = std::false_type;
    if (ids)
        drop ? run(T_{}, T_{}) : run(T_{}, F_{});
    else
        drop ? run(F_{}, T_{}) : run(F_{}, F_{});
    if (hipGetLastError() != hipSuccess) return false;
    return launch_colsum(pg, nblk, D, dg, c.ws + c.w.colsum, c.stream) == hipSuccess &&
           launch_colsum(pb, nblk, D, db, c.ws + c.w.colsum, c.stream) == hipSuccess;
}

template <int NV>
int train_step_t(const Dims& d, const StepOpts& o, const float* params, const int* ids,
                 const int* targets, float* grads, float* loss, char* ws, const Layout& w,
                 rocblas_handle blas, hipStream_t stream) {
    Ctx c{blas, stream, ws, w};
    const int64_t B = d.B, T = d.T, M = B * T, D = d.D, ED = d.E * d.D, F = 4 * d.D, V = d.V;
    const int64_t nt = tensor_count(d);
    int64_t off[3 + kLayerTensors * 64];
    if (nt > (int64_t)(sizeof(off) / sizeof(off[0]))) return RECBLR_ERR_UNSUPPORTED;
    param_offsets(d, off);
    auto P = [&](int64_t l, int k) { return params + off[3 + l * kLayerTensors + k]; };
    auto G = [&](int64_t l, int k) { return grads + off[3 + l * kLayerTensors + k]; };
    auto buf = [&](size_t o) { return (float*)(ws + o); };
    float* H = buf(w.H);
    auto Hl = [&](int64_t l) { return H + l * M * D; };
    auto per = [&](size_t o, int64_t l, int64_t width) { return buf(o) + l * M * width; };
    float* st = buf(w.stats);
    auto stat = [&](int64_t l, int k) { return st + (l * 4 + k) * M; };
    float* mu0 = buf(w.emb_stats);
    float* rs0 = mu0 + M;
    const float* E = params + off[0];
    if (rocblas_set_stream(blas, stream) != rocblas_status_success) return RECBLR_ERR_HIP;
    int st_ = RECBLR_OK;
#define CHECK(x) \
    do {         \
        if (!(x)) return RECBLR_ERR_HIP; \
    } while (0)
#define CHECK_ST(x)                  \
    do {                             \
        if ((st_ = (x)) != RECBLR_OK) return st_; \
    } while (0)

    // ---- dropout masks: every site's keep bits, drawn once for the step
    const bool dropout = o.dropout > 0.0f;
    const int64_t mwords = mask_words(d);
    uint32_t* mask = (uint32_t*)(ws + w.mask);
    auto site = [&](int64_t k, int pad = -1) {
        Drop dr;
        dr.pad = pad;
        if (dropout) {
            dr.keep = mask + k * mwords;
            dr.scale = 1.0f / (1.0f - o.dropout);
        }
        return dr;
    };
    if (dropout) {
        const int64_t total = mask_sites(d) * mwords;
        const uint32_t thr = (uint32_t)floor((double)o.dropout * 4294967296.0);
        hipLaunchKernelGGL(dropout_mask_kernel, dim3(blocks_for(total)), dim3(kThreads), 0,
                           stream, mask, mwords, total, thr, o.seed, o.offset);
        CHECK(hipGetLastError() == hipSuccess);
    }
    float* Z = buf(w.Z);

    // ---- forward
    CHECK(ln_fwd<NV>(c, E, nullptr, ids, params + off[1], params + off[2], nullptr, Hl(0), mu0,
                     rs0, M, V, d.eps, site(0, o.pad_id)));
    for (int64_t l = 0; l < d.layers; ++l) {
        float *Hx = per(w.Hx, l, ED), *Hz = per(w.Hz, l, ED), *hb = per(w.hb, l, ED),
              *y = per(w.y, l, ED), *s1 = per(w.s1, l, D), *H1 = per(w.H1, l, D),
              *A = per(w.A, l, F), *Pp = per(w.P, l, F), *s2 = per(w.s2, l, D);
        CHECK(linear_fwd(c, Hl(l), P(l, kWx), P(l, kbx), Hx, M, ED, D));
        CHECK(linear_fwd(c, Hl(l), P(l, kWz), P(l, kbz), Hz, M, ED, D));
        CHECK_ST(recblr_gated_forward(Hx, Hz, P(l, kConvW), P(l, kConvB), d.K, P(l, kWr),
                                      P(l, kbr), P(l, kWi), P(l, kbi), P(l, kLam), nullptr, y, hb,
                                      nullptr, B, T, ED, RECBLR_F32, ws + w.gated, w.gated_bytes,
                                      stream));
        // O = y Wo^T + bo goes to s1, then s1 += H and H1 = LN(s1).
        CHECK(linear_fwd(c, y, P(l, kWo), P(l, kbo), s1, M, D, ED));
        CHECK(ln_fwd<NV>(c, s1, Hl(l), nullptr, P(l, kLn1g), P(l, kLn1b), s1, H1, stat(l, 0),
                         stat(l, 1), M, V, d.eps, site(1 + 2 * l)));
        CHECK(linear_fwd(c, H1, P(l, kW1), P(l, kb1), A, M, F, D, Pp));  // Pp = SiLU(A)
        CHECK(linear_fwd(c, Pp, P(l, kW2), P(l, kb2), s2, M, D, F));
        CHECK(ln_fwd<NV>(c, s2, H1, nullptr, P(l, kLn2g), P(l, kLn2b), s2, Hl(l + 1),
                         stat(l, 2), stat(l, 3), M, V, d.eps, site(2 + 2 * l)));
    }
    // prediction: logits = h_T E^T with h_T the last step of every row
    const float* hT = Hl(d.layers) + (T - 1) * D;
    float* logits = buf(w.logits);
    float* dlogits = buf(w.dlogits);
    CHECK(gemm_xwT(c, hT, T * D, E, logits, V, B, V, D, 0.0f));
    hipLaunchKernelGGL(ce_kernel, dim3((unsigned)B), dim3(kThreads), 0, stream, logits, targets, B,
                       V, dlogits, buf(w.lossb));
    CHECK(hipGetLastError() == hipSuccess);
    hipLaunchKernelGGL(loss_final_kernel, dim3(1), dim3(kThreads), 0, stream, buf(w.lossb), B,
                       loss);
    CHECK(hipGetLastError() == hipSuccess);

    // ---- backward
    float *X = buf(w.X), *Y = buf(w.Y), *dP = buf(w.dP), *dY = buf(w.dY), *dHx = buf(w.dHx),
          *dHz = buf(w.dHz);
    float* dE = grads + off[0];
    // dE = dlogits^T h_T (the prediction's use of E); the input side adds on later.
    CHECK(gemm_dyTx(c, hT, T * D, dlogits, V, dE, B, V, D));
    // dH of the last layer's output: zero except the last step, dlogits E.
    CHECK(launch_fill(Y, 0.0f, M * D, stream) == hipSuccess);
    CHECK(gemm_dyW(c, dlogits, V, E, Y + (T - 1) * D, T * D, B, V, D, 0.0f));
    for (int64_t l = d.layers - 1; l >= 0; --l) {
        float *Hx = per(w.Hx, l, ED), *Hz = per(w.Hz, l, ED), *hb = per(w.hb, l, ED),
              *y = per(w.y, l, ED), *s1 = per(w.s1, l, D), *H1 = per(w.H1, l, D),
              *A = per(w.A, l, F), *Pp = per(w.P, l, F), *s2 = per(w.s2, l, D);
        // LN2: Y (dH2) -> X (ds2: the residual part of dH1) and dQ (ds2 through
        // the dropout, in Z; X itself without dropout)
        float* dQ = dropout ? Z : X;
        CHECK(ln_bwd<NV>(c, Y, s2, nullptr, stat(l, 2), stat(l, 3), P(l, kLn2g), X, G(l, kLn2g),
                         G(l, kLn2b), M, V, site(2 + 2 * l), dropout ? Z : nullptr));
        // PFFN: Q = P W2^T + b2, P = SiLU(A), A = H1 W1^T + b1
        CHECK(linear_wgrad(c, Pp, dQ, G(l, kW2), G(l, kb2), M, D, F));
        // dP = (dQ W2) * SiLU'(A)
        CHECK(linear_dgrad(c, dQ, P(l, kW2), dP, M, D, F, LinearMode::kSiluGrad, A));
        CHECK(linear_wgrad(c, H1, dP, G(l, kW1), G(l, kb1), M, F, D));
        CHECK(linear_dgrad(c, dP, P(l, kW1), X, M, F, D, LinearMode::kAccumulate));  // X = dH1
        // LN1: X (dH1) -> Y (ds1: the residual part of dH) and dO (ds1 through
        // the dropout, in Z; Y itself without dropout)
        float* dO = dropout ? Z : Y;
        CHECK(ln_bwd<NV>(c, X, s1, nullptr, stat(l, 0), stat(l, 1), P(l, kLn1g), Y, G(l, kLn1g),
                         G(l, kLn1b), M, V, site(1 + 2 * l), dropout ? Z : nullptr));
        // O = y Wo^T + bo
        CHECK(linear_wgrad(c, y, dO, G(l, kWo), G(l, kbo), M, D, ED));
        CHECK(linear_dgrad(c, dO, P(l, kWo), dY, M, D, ED, LinearMode::kStore));
        CHECK_ST(recblr_gated_backward(Hx, Hz, P(l, kConvW), P(l, kConvB), d.K, P(l, kWr),
                                       P(l, kbr), P(l, kWi), P(l, kbi), P(l, kLam), nullptr, hb,
                                       dY, nullptr, dHx, dHz, G(l, kConvW), G(l, kConvB),
                                       G(l, kWr), G(l, kbr), G(l, kWi), G(l, kbi), G(l, kLam),
                                       nullptr, B, T, ED, RECBLR_F32, ws + w.gated, w.gated_bytes,
                                       stream));
        // Hx = H Wx^T + bx, Hz = H Wz^T + bz; Y becomes dH of this layer's input.
        CHECK(linear_wgrad(c, Hl(l), dHx, G(l, kWx), G(l, kbx), M, ED, D));
        CHECK(linear_wgrad(c, Hl(l), dHz, G(l, kWz), G(l, kbz), M, ED, D));
        CHECK(linear_dgrad(c, dHx, P(l, kWx), Y, M, ED, D, LinearMode::kAccumulate));
        CHECK(linear_dgrad(c, dHz, P(l, kWz), Y, M, ED, D, LinearMode::kAccumulate));
    }
    // embedding LayerNorm, then the input side of dE: rows summed per item
    CHECK(ln_bwd<NV>(c, Y, E, ids, mu0, rs0, params + off[1], X, grads + off[1], grads + off[2], M,
                     V, site(0, o.pad_id)));
    unsigned* ids_s = (unsigned*)(ws + w.ids_s);
    int* pos = (int*)(ws + w.pos);
    int* pos_s = (int*)(ws + w.pos_s);
    hipLaunchKernelGGL(iota_kernel, dim3(blocks_for(M)), dim3(kThreads), 0, stream, pos, M);
    CHECK(hipGetLastError() == hipSuccess);
    size_t sb = w.sort_bytes;
    CHECK(hipcub::DeviceRadixSort::SortPairs(ws + w.sort_tmp, sb, (const unsigned*)ids, ids_s,
                                             (const int*)pos, pos_s, (int)M, 0, 32,
                                             stream) == hipSuccess);
    int64_t* lo = (int64_t*)(ws + w.emb_lo);
    int64_t* hi = (int64_t*)(ws + w.emb_hi);
    int64_t* np_ = (int64_t*)(ws + w.emb_np);
    int64_t* poff = (int64_t*)(ws + w.emb_poff);
    float* epart = buf(w.emb_part);
    const int64_t max_pieces = (M + kPiece - 1) / kPiece + V;
    hipLaunchKernelGGL(emb_count_kernel, dim3(blocks_for(V)), dim3(kThreads), 0, stream, ids_s, M,
                       V, lo, hi, np_);
    CHECK(hipGetLastError() == hipSuccess);
    hipLaunchKernelGGL(exclusive_scan_kernel, dim3(1), dim3(1024), 0, stream, np_, poff, V);
    CHECK(hipGetLastError() == hipSuccess);
    hipLaunchKernelGGL((emb_piece_kernel<NV>), dim3(blocks_for(max_pieces, 4)), dim3(kThreads), 0,
                       stream, pos_s, X, lo, hi, poff, epart, V, max_pieces);
    CHECK(hipGetLastError() == hipSuccess);
    hipLaunchKernelGGL((emb_item_kernel<NV>), dim3(blocks_for(V, 4)), dim3(kThreads), 0, stream,
                       poff, epart, dE, V);
    CHECK(hipGetLastError() == hipSuccess);
#undef CHECK
#undef CHECK_ST
    return RECBLR_OK;
}

}  // namespace

int train_step(const Dims& d, const StepOpts& o, const float* params, const int* ids,
               const int* targets, float* grads, float* loss, void* ws, rocblas_handle blas,
               hipStream_t stream) {
    const Layout w = layout(d);
    // Padding between tensors is zero in the gradient.
    if (launch_fill(grads, 0.0f, param_offsets(d, nullptr), stream) != hipSuccess)
        return RECBLR_ERR_HIP;
    char* wsb = (char*)ws;
    switch (d.D / 64) {
        case 1: return train_step_t<1>(d, o, params, ids, targets, grads, loss, wsb, w, blas, stream);
        case 2: return train_step_t<2>(d, o, params, ids, targets, grads, loss, wsb, w, blas, stream);
        case 4: return train_step_t<4>(d, o, params, ids, targets, grads, loss, wsb, w, blas, stream);
        default: return RECBLR_ERR_UNSUPPORTED;
    }
}

hipError_t adam(float* p, const float* g, float* m1, float* m2, int64_t n, int64_t step, float lr,
                float b1, float b2, float eps, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    const float c1 = 1.0f - powf(b1, (float)step), c2 = 1.0f - powf(b2, (float)step);
    hipLaunchKernelGGL(adam_kernel, dim3(blocks_for(n)), dim3(kThreads), 0, stream, p, g, m1, m2,
                       n, lr, b1, b2, eps, c1, c2);
    return hipGetLastError();
}

}  // namespace model
}  // namespace recblr
