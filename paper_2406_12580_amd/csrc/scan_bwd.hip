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
// Decomposition mirrors the forward kernels (lane = VEC channels, W waves per
// macro-chunk of W*C steps): the chain kernel walks the macro-chunks from the
// end of the sequence to its start; the look-back kernel hands out tiles from
// the end too, so that tile index r in processing order is macro-chunk
// nseg-1-r and the forward look-back code applies unchanged.
#include "device_common.hpp"
#include "fused_z.hpp"
#include "launch.hpp"
#include "lookback.hpp"

namespace recblr {

namespace {

constexpr size_t kAlign = 256;
inline size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// Rows of the per-channel dLambda partials are reduced in blocks of this many.
constexpr int kReduceRows = 64;

}  // namespace

struct BwdParams {
    const void* x;
    const void* zr;
    const void* zi;
    const float* lam;
    const float* h0;
    const void* h;
    const void* dh;
    const float* dhT;
    void* dx;
    void* dzr;
    void* dzi;
    float* dh0;
    float* partial;  // [nseg][B*D] per-tile sums of dLoss/dq * r
    int64_t L, D, nch;
    int64_t ngroups, nseg;
    LookbackWs lb;
    unsigned* dl_counters;  // one per 64-channel column group of the dLambda reduction
    int64_t n_counters;
    // Fused kernel only, fp32 x: when gy is set, dh is not read but formed on
    // load as dh_t = gy_t SiLU(gz_t) (the output gate of the gated layer), in
    // fp32; with fp32 h, if gdz is set too, the gate input's gradient
    // gy_t h_t SiLU'(gz_t) is stored there (same layout as h).
    const void* gy = nullptr;
    const void* gz = nullptr;
    void* gdz = nullptr;
};

// Zeroes the dLambda counters (n of them); called by one workgroup of each
// backward scan kernel, which runs before the reduction.
__device__ __forceinline__ void zero_counters(unsigned* c, int64_t n) {
    for (int64_t i = threadIdx.x; i < n; i += blockDim.x) c[i] = 0u;
}

template <typename TX, int VEC, typename Off>
struct BwdLane {
    bool valid;
    int64_t c0, d0;
    Off base, row;
    __device__ __forceinline__ void init(int64_t group, int lane, int64_t L, int64_t D,
                                         int64_t nch) {
        const int64_t c = (group * kWave + lane) * VEC;
        valid = c < nch;
        c0 = valid ? c : 0;  // idle lanes shadow channel 0 and store nothing
        const int64_t b = c0 / D;
        d0 = c0 - b * D;
        base = (Off)((b * L * D + d0) * (int64_t)sizeof(TX));
        row = (Off)(D * (int64_t)sizeof(TX));
    }
    __device__ __forceinline__ Off at(int64_t t) const { return base + (Off)t * row; }
};

// Raw inputs of C steps (clamped to L-1; masked later), h_{t-1} for each of
// them (h0 at t = 0) and z_r of the step right after the chunk.
template <typename TX, typename TZ, int C, int VEC, typename Off>
struct BwdIn {
    float g[C][VEC], x[C][VEC], zr[C][VEC], zi[C][VEC], hp[C][VEC];
    float zr_after[VEC];

    // FULL: 0 < t and t + 1 < L for every step of the chunk (no clamping, no h0).
    template <bool FULL>
    __device__ __forceinline__ void fetch(const BwdParams& P, const BwdLane<TX, VEC, Off>& ln,
                                          const float (&h0v)[VEC], int64_t t_first) {
#pragma unroll
        for (int j = 0; j < C; ++j) {
            const int64_t t = FULL || t_first + j < P.L ? t_first + j : P.L - 1;
            const Off off = ln.at(t);
            load_vec<TX, VEC>((const TX*)P.dh, off, g[j]);
            load_vec<TX, VEC>((const TX*)P.x, off, x[j]);
            load_vec<TZ, VEC>((const TZ*)P.zr, z_offset<TX, TZ>(off), zr[j]);
            load_vec<TZ, VEC>((const TZ*)P.zi, z_offset<TX, TZ>(off), zi[j]);
            load_vec<TX, VEC>((const TX*)P.h, FULL || t > 0 ? off - ln.row : off, hp[j]);
            if (!FULL && t == 0) {
#pragma unroll
                for (int k = 0; k < VEC; ++k) hp[j][k] = h0v[k];
            }
        }
        const int64_t ta = FULL || t_first + C < P.L ? t_first + C : P.L - 1;
        load_vec<TZ, VEC>((const TZ*)P.zr, z_offset<TX, TZ>(ln.at(ta)), zr_after);
    }
};

// Step pairs are stored for fp32 I/O and formed on use for bf16 I/O (the
// faster choice for each on MI355X).
template <typename TX>
constexpr bool kKeepPairs = sizeof(TX) == 4;

// Per-step pieces of the reverse recurrence kept in registers: r_t and
// alpha_t of every step of the chunk, alpha of the step right after it, and
// the pair (alpha_{t+1}, G_t) of every step (identity (1, 0) past the end,
// alpha_{L+1} = 0, dhT added at t = L-1).  With KEEP the pairs are stored
// once; without, each is formed where it is used, which saves two registers
// per step (bf16 I/O: 126 instead of 160 VGPRs at 12 steps per wave, so two
// 8-wave workgroups fit on a compute unit).
template <int C, int VEC, bool KEEP>
struct BwdSteps {
    float r[C][VEC], al[C][VEC], al_after[VEC], dhT[VEC];
    float ap[KEEP ? C : 1][VEC], gg[KEEP ? C : 1][VEC];
    int64_t t_first, L;

    template <bool FULL>
    __device__ __forceinline__ Seg form_pair(const float (&g)[VEC], int j, int k) const {
        const float nxt = j + 1 < C ? al[j + 1 < C ? j + 1 : j][k] : al_after[k];
        if (FULL) return Seg{nxt, g[k]};
        const int64_t t = t_first + j;
        const float gj = g[k] + (t == L - 1 ? dhT[k] : 0.0f);
        return Seg{t < L ? (t + 1 < L ? nxt : 0.0f) : 1.0f, t < L ? gj : 0.0f};
    }
    template <bool FULL>
    __device__ __forceinline__ Seg pair(const float (&g)[VEC], int j, int k) const {
        if constexpr (KEEP) return Seg{ap[KEEP ? j : 0][k], gg[KEEP ? j : 0][k]};
        else return form_pair<FULL>(g, j, k);
    }
};

template <bool FULL, typename TX, typename TZ, int C, int VEC, typename Off, bool KEEP>
__device__ __forceinline__ void form_bwd(const BwdIn<TX, TZ, C, VEC, Off>& in,
                                         const ChannelConst (&cc)[VEC], const float (&dhTv)[VEC],
                                         int64_t t_first, int64_t L,
                                         BwdSteps<C, VEC, KEEP>& st) {
#pragma unroll
    for (int j = 0; j < C; ++j)
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
            st.r[j][k] = sigmoid(in.zr[j][k]);
            st.al[j][k] = fast_exp2(st.r[j][k] * cc[k].neg_s_l2);
        }
#pragma unroll
    for (int k = 0; k < VEC; ++k) {
        st.al_after[k] = fast_exp2(sigmoid(in.zr_after[k]) * cc[k].neg_s_l2);
        st.dhT[k] = dhTv[k];
    }
    st.t_first = t_first;
    st.L = L;
    if constexpr (KEEP) {
#pragma unroll
        for (int j = 0; j < C; ++j)
#pragma unroll
            for (int k = 0; k < VEC; ++k) {
                const Seg p = st.template form_pair<FULL>(in.g[j], j, k);
                st.ap[KEEP ? j : 0][k] = p.A;
                st.gg[KEEP ? j : 0][k] = p.H;
            }
    }
}

template <bool FULL, typename TX, typename TZ, int C, int VEC, typename Off, bool KEEP>
__device__ __forceinline__ void local_reverse(const BwdIn<TX, TZ, C, VEC, Off>& in,
                                              const BwdSteps<C, VEC, KEEP>& st, Seg (&s)[VEC]) {
#pragma unroll
    for (int k = 0; k < VEC; ++k) {
        s[k] = Seg{1.0f, 0.0f};
#pragma unroll
        for (int j = C - 1; j >= 0; --j) s[k] = compose(st.template pair<FULL>(in.g[j], j, k), s[k]);
    }
}

// Run the chunk backwards from delta (the adjoint right after the chunk) and
// apply the gate-gradient epilogue to every step before L.  GROUPED: the
// gradient terms share dLoss/dq = -alpha g_alpha + g_beta i alpha^2 /
// sqrt(1 - alpha^2) (dLambda adds r dLoss/dq, dz_r = s r (1 - r) dLoss/dq),
// four vector instructions fewer per element; the look-back kernels take it
// (256 x 2048 x 128 fp32 backward 362-365 -> 358 us), while the chain kernel
// keeps the two terms apart (with the grouped form its 2048 x 200 x 64
// backward measured 154-157 against 148-151 us).
template <bool FULL, bool GROUPED, typename TX, typename TZ, int C, int VEC, typename Off, bool KEEP>
__device__ __forceinline__ void emit_bwd(const BwdParams& P, const BwdLane<TX, VEC, Off>& ln,
                                         const BwdIn<TX, TZ, C, VEC, Off>& in,
                                         const BwdSteps<C, VEC, KEEP>& st,
                                         const ChannelConst (&cc)[VEC], int64_t t_first,
                                         float (&delta)[VEC], float (&dsum)[VEC]) {
#pragma unroll
    for (int j = C - 1; j >= 0; --j) {
        const int64_t t = t_first + j;
        float dxv[VEC], dzrv[VEC], dziv[VEC];
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
            const Seg pj = st.template pair<FULL>(in.g[j], j, k);
            delta[k] = fmaf(pj.A, delta[k], pj.H);
            const float r = st.r[j][k], al = st.al[j][k];
            const float i = sigmoid(in.zi[j][k]);
            const float mm = one_minus_exp_neg(r * cc[k].two_s, al);
            const float rs = mm > 0.0f ? fast_rsq(mm) : 0.0f;
            const float sq = mm * rs;  // sqrt(1 - alpha^2)
            if constexpr (!GROUPED) {
            const float q = r * cc[k].s;
            const float g_alpha = delta[k] * in.hp[j][k];
            const float g_beta = delta[k] * in.x[j][k];
            const float g1 = -al * g_alpha;
            const float g2 = g_beta * i * al * al;
            if (FULL || t < P.L) dsum[k] = fmaf(g1, r, fmaf(g2, r * rs, dsum[k]));
            dxv[k] = delta[k] * sq * i;
            dzrv[k] = fmaf(g1, q, g2 * (q * rs)) * (1.0f - r);
            dziv[k] = g_beta * sq * i * (1.0f - i);
            } else {
            const float g_alpha = delta[k] * in.hp[j][k];
            const float gbi = delta[k] * in.x[j][k] * i;  // dLoss/dbeta * i
            // dLoss/dq = -alpha g_alpha + g_beta i alpha^2 / sqrt(1 - alpha^2)
            const float gq = fmaf(gbi * (al * al), rs, -al * g_alpha);
            if (FULL || t < P.L) dsum[k] = fmaf(gq, r, dsum[k]);
            dxv[k] = delta[k] * (sq * i);
            dzrv[k] = gq * (cc[k].s * fmaf(-r, r, r));  // dq/dz_r = s r (1 - r)
            dziv[k] = gbi * sq * (1.0f - i);
            }
        }
        if (ln.valid && (FULL || t < P.L)) {
            const Off off = ln.at(t);
            store_vec<TX, VEC>((TX*)P.dx, off, dxv);
            store_vec<TZ, VEC>((TZ*)P.dzr, z_offset<TX, TZ>(off), dzrv);
            store_vec<TZ, VEC>((TZ*)P.dzi, z_offset<TX, TZ>(off), dziv);
            if (!FULL && t == 0 && P.dh0) {
#pragma unroll
                for (int k = 0; k < VEC; ++k) P.dh0[ln.c0 + k] = st.al[j][k] * delta[k];
            }
        }
    }
}

template <int VEC>
__device__ __forceinline__ void bwd_lane_consts(const BwdParams& P, int64_t c0, int64_t d0,
                                                ChannelConst (&cc)[VEC], float (&h0v)[VEC],
                                                float (&dhTv)[VEC]) {
#pragma unroll
    for (int k = 0; k < VEC; ++k) {
        cc[k] = channel_const(P.lam[d0 + k]);
        h0v[k] = P.h0 ? P.h0[c0 + k] : 0.0f;
        dhTv[k] = P.dhT ? P.dhT[c0 + k] : 0.0f;
    }
}

// Sum the waves' dLambda partials of this workgroup in a fixed order.
template <int W, int VEC>
__device__ __forceinline__ void write_partial(float (&red)[W][kWave][VEC],
                                              const float (&dsum)[VEC], float* out, bool valid,
                                              int w, int lane) {
#pragma unroll
    for (int k = 0; k < VEC; ++k) red[w][lane][k] = dsum[k];
    __syncthreads();
    if (w == 0 && valid) {
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
            float acc = 0.0f;
#pragma unroll
            for (int q = 0; q < W; ++q) acc += red[q][lane][k];
            out[k] = acc;
        }
    }
}

// ------------------------------------------------------------------ chain kernel
// One macro-chunk, backwards: reverse local aggregates through LDS, carry fold
// from the later waves, gate-gradient epilogue and stores.
template <bool FULL, typename TX, typename TZ, int W, int C, int VEC, typename Off>
__device__ __forceinline__ void chain_bwd_step(const BwdParams& P, const BwdLane<TX, VEC, Off>& ln,
                                               const BwdIn<TX, TZ, C, VEC, Off>& cur,
                                               const ChannelConst (&cc)[VEC],
                                               const float (&dhTv)[VEC],
                                               Seg (&agg)[W][kWave][VEC], int64_t tw, int w,
                                               int lane, float (&carry)[VEC],
                                               float (&dsum)[VEC]) {
    BwdSteps<C, VEC, kKeepPairs<TX>> st;
    form_bwd<FULL>(cur, cc, dhTv, tw, P.L, st);
    Seg s[VEC];
    local_reverse<FULL>(cur, st, s);
#pragma unroll
    for (int k = 0; k < VEC; ++k) agg[w][lane][k] = s[k];
    __syncthreads();
    // Carry into this wave: the later waves, last one first.
    float delta[VEC], cout[VEC];
#pragma unroll
    for (int k = 0; k < VEC; ++k) delta[k] = carry[k];
#pragma unroll
    for (int q = W - 1; q >= 0; --q) {
        if (q > w) {
#pragma unroll
            for (int k = 0; k < VEC; ++k) {
                const Seg e = agg[q][lane][k];
                delta[k] = fmaf(e.A, delta[k], e.H);
            }
        }
    }
#pragma unroll
    for (int k = 0; k < VEC; ++k) cout[k] = delta[k];
    emit_bwd<FULL, false>(P, ln, cur, st, cc, tw, delta, dsum);
    // Carry out of the macro-chunk, towards earlier steps.
#pragma unroll
    for (int q = W - 1; q >= 0; --q) {
        if (q <= w) {
#pragma unroll
            for (int k = 0; k < VEC; ++k) {
                const Seg e = agg[q][lane][k];
                cout[k] = fmaf(e.A, cout[k], e.H);
            }
        }
    }
#pragma unroll
    for (int k = 0; k < VEC; ++k) carry[k] = cout[k];
}

// Macro-chunks are walked from the end of the sequence.  The first one
// processed (holding t = L-1) and the last (holding t = 0) take the masked
// path; the steady-state loop in between has no branch around a memory
// instruction (see the forward chain kernel) and always prefetches the next
// chunk.
template <typename TX, typename TZ, int W, int C, int VEC, typename Off>
__global__ __launch_bounds__(W* kWave) void scan_bwd_chain_kernel(BwdParams P) {
    __shared__ Seg agg[2][W][kWave][VEC];
    __shared__ float red[W][kWave][VEC];
    const int lane = threadIdx.x & (kWave - 1);
    const int w = wave_id();
    if (blockIdx.x == 0) {
        zero_counters(P.dl_counters, P.n_counters);
        if (threadIdx.x == 0 && P.lb.status) *P.lb.status = 0u;  // no waits in this kernel
    }
    BwdLane<TX, VEC, Off> ln;
    ln.init(blockIdx.x, lane, P.L, P.D, P.nch);
    ChannelConst cc[VEC];
    float h0v[VEC], dhTv[VEC], carry[VEC], dsum[VEC];
    bwd_lane_consts<VEC>(P, ln.c0, ln.d0, cc, h0v, dhTv);
#pragma unroll
    for (int k = 0; k < VEC; ++k) carry[k] = dsum[k] = 0.0f;

    constexpr int64_t kMacro = (int64_t)W * C;
    const int64_t nmacro = (P.L + kMacro - 1) / kMacro;
    const int64_t woff = (int64_t)w * C;
    // Two buffers alternate roles (loop unrolled by two), so no register copy
    // ties the prefetched chunk to the one being consumed.
    BwdIn<TX, TZ, C, VEC, Off> bufA, bufB;
    if (nmacro > 0) {
        int64_t m = nmacro - 1;
        bufA.template fetch<false>(P, ln, h0v, m * kMacro + woff);
        if (m == 0) {
            chain_bwd_step<false>(P, ln, bufA, cc, dhTv, agg[0], woff, w, lane, carry, dsum);
        } else {
            bufB.template fetch<false>(P, ln, h0v, (m - 1) * kMacro + woff);
            chain_bwd_step<false>(P, ln, bufA, cc, dhTv, agg[m & 1], m * kMacro + woff, w, lane,
                                  carry, dsum);
            --m;
            for (;;) {
                if (m == 0) {
                    chain_bwd_step<false>(P, ln, bufB, cc, dhTv, agg[0], woff, w, lane, carry, dsum);
                    break;
                }
                bufA.template fetch<false>(P, ln, h0v, (m - 1) * kMacro + woff);
                chain_bwd_step<true>(P, ln, bufB, cc, dhTv, agg[m & 1], m * kMacro + woff, w,
                                     lane, carry, dsum);
                --m;
                if (m == 0) {
                    chain_bwd_step<false>(P, ln, bufA, cc, dhTv, agg[0], woff, w, lane, carry, dsum);
                    break;
                }
                bufB.template fetch<false>(P, ln, h0v, (m - 1) * kMacro + woff);
                chain_bwd_step<true>(P, ln, bufA, cc, dhTv, agg[m & 1], m * kMacro + woff, w,
                                     lane, carry, dsum);
                --m;
            }
        }
    }
    if (P.L == 0 && w == 0 && ln.valid && P.dh0) {
#pragma unroll
        for (int k = 0; k < VEC; ++k) P.dh0[ln.c0 + k] = dhTv[k];
    }
    write_partial<W, VEC>(red, dsum, P.partial + ln.c0, ln.valid, w, lane);
}

// ------------------------------------------------------------------ look-back kernel
template <typename TX, typename TZ, int W, int C, int VEC, int K, typename Off>
__global__ __launch_bounds__(W* kWave) void scan_bwd_lookback_kernel(BwdParams P) {
    __shared__ Seg agg[W][kWave][VEC];
    __shared__ uint64_t win_sh[W * K][kWave][VEC];
    __shared__ float carry_sh[kWave][VEC];
    __shared__ float red[W][kWave][VEC];
    __shared__ int64_t tile_sh;
    const int lane = threadIdx.x & (kWave - 1);
    const int w = wave_id();
    if (threadIdx.x == 0) tile_sh = (int64_t)atomicAdd(P.lb.ticket, 1u);
    __syncthreads();
    const int64_t tile = tile_sh;
    if (tile >= P.ngroups * P.nseg) return;  // only if the workspace was shared by two calls
    const int64_t r = tile / P.ngroups;  // processing order: from the end of the sequence
    const int64_t g = tile - r * P.ngroups;
    const int64_t s = P.nseg - 1 - r;    // macro-chunk of this tile
    if (tile == 0) zero_counters(P.dl_counters, P.n_counters);

    BwdLane<TX, VEC, Off> ln;
    ln.init(g, lane, P.L, P.D, P.nch);
    ChannelConst cc[VEC];
    float h0v[VEC], dhTv[VEC], dsum[VEC], zero[VEC];
    bwd_lane_consts<VEC>(P, ln.c0, ln.d0, cc, h0v, dhTv);
#pragma unroll
    for (int k = 0; k < VEC; ++k) dsum[k] = zero[k] = 0.0f;

    const int64_t tw = s * W * C + (int64_t)w * C;
    const bool full = s > 0 && (s + 1) * W * C < P.L;  // workgroup-uniform
    BwdIn<TX, TZ, C, VEC, Off> in;
    BwdSteps<C, VEC, kKeepPairs<TX>> st;
    if (full) {
        in.template fetch<true>(P, ln, h0v, tw);
        form_bwd<true>(in, cc, dhTv, tw, P.L, st);
    } else {
        in.template fetch<false>(P, ln, h0v, tw);
        form_bwd<false>(in, cc, dhTv, tw, P.L, st);
    }
    {
        Seg sg[VEC];
        if (full) local_reverse<true>(in, st, sg);
        else local_reverse<false>(in, st, sg);
#pragma unroll
        for (int k = 0; k < VEC; ++k) agg[w][lane][k] = sg[k];
    }
    __syncthreads();
    // pre: the waves after this one (applied first); tot: the whole tile.
    Seg pre[VEC], tot[VEC];
#pragma unroll
    for (int k = 0; k < VEC; ++k) pre[k] = tot[k] = Seg{1.0f, 0.0f};
#pragma unroll
    for (int q = W - 1; q >= 0; --q) {
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
            const Seg e = agg[q][lane][k];
            if (q > w) pre[k] = compose(e, pre[k]);
            tot[k] = compose(e, tot[k]);
        }
    }
    __syncthreads();  // agg is reused below

    uint64_t* const own = P.lb.states + r * P.nch + ln.c0;
    if (r == 0) {
        if (w == 0) {
#pragma unroll
            for (int k = 0; k < VEC; ++k) {
                carry_sh[lane][k] = 0.0f;
                if (ln.valid) publish(own + k, pack_inclusive(tot[k].H));
            }
        }
    } else {
        if (w == 0 && ln.valid) {
#pragma unroll
            for (int k = 0; k < VEC; ++k) publish(own + k, pack_aggregate(tot[k]));
        }
        lookback_carry<W, VEC, K>(P.lb.states, P.nch, ln.c0, r, zero, win_sh, carry_sh, w, lane,
                           P.lb.status);
        if (w == 0 && ln.valid) {
#pragma unroll
            for (int k = 0; k < VEC; ++k)
                publish(own + k, pack_inclusive(fmaf(tot[k].A, carry_sh[lane][k], tot[k].H)));
        }
    }
    __syncthreads();
    float delta[VEC];
#pragma unroll
    for (int k = 0; k < VEC; ++k) delta[k] = fmaf(pre[k].A, carry_sh[lane][k], pre[k].H);
    if (full) emit_bwd<true, true>(P, ln, in, st, cc, tw, delta, dsum);
    else emit_bwd<false, true>(P, ln, in, st, cc, tw, delta, dsum);
    write_partial<W, VEC>(red, dsum, P.partial + s * P.nch + ln.c0, ln.valid, w, lane);
}

// ------------------------------------------------------------------ projections fused in
// The layer backward's scan: a look-back kernel that recomputes its own gate
// pre-activations on the matrix cores (fused_z.hpp) instead of reading z, so
// the layer backward does not project x once more through HBM.  The adjoint
// runs in the form
//   eps_t = alpha_t (G_t + eps_{t+1}),   eps_L = dhT,   delta_t = G_t + eps_{t+1},
// (eps_t = alpha_t delta_t is what flows from step t into h_{t-1}), whose
// per-step pair (alpha_t, alpha_t G_t) belongs to step t alone: a tile needs
// no z of the step after it.  dh0 = eps_0.  The epilogue is that of emit_bwd.
// x: [B][L][D] I/O type; dx is written in the I/O type, dz_r, dz_i in fp32.
// A wave's C rows (steps) of its 64 channels of one tensor, staged into LDS
// with 16-byte direct-to-LDS loads (the channels of a wave are contiguous
// because D % 64 == 0): step j of lane l lands at ((T*)dst)[j * 64 + l].
// Rows are t_first + shift + j, clamped to [0, L-1].
template <typename T, int C>
__device__ __forceinline__ void stage_rows(const T* tensor, int64_t b, int64_t L, int64_t D,
                                           int64_t dg, int64_t t_first, int shift, char* dst,
                                           int lane) {
    constexpr int kRow = kWave * (int)sizeof(T);  // bytes of one step's 64 channels
    constexpr int kLanesPerRow = kRow / 16;
    constexpr int kRowsPerLoad = kWave / kLanesPerRow;
    static_assert(C % kRowsPerLoad == 0, "whole loads per wave");
    const int64_t col = (int64_t)(lane % kLanesPerRow) * (16 / (int)sizeof(T));
#pragma unroll
    for (int i = 0; i < C / kRowsPerLoad; ++i) {
        int64_t t = t_first + shift + i * kRowsPerLoad + lane / kLanesPerRow;
        t = t < 0 ? 0 : (t < L ? t : L - 1);
        const T* gp = tensor + (b * L + t) * D + dg + col;
        __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)gp,
                                         (__attribute__((address_space(3))) void*)(dst + i * 1024),
                                         16, 0, 0);
    }
}

template <typename T>
__device__ __forceinline__ float lds_elem(const char* base, int idx) {
    if constexpr (sizeof(T) == 4) return ((const float*)base)[idx];
    else return __uint_as_float((uint32_t)((const uint16_t*)base)[idx] << 16);
}

// One backward tile in the eps form, from its gate pre-activations: zr, zi
// hold the lane's channel at this wave's C steps (tile row s = nseg-1-r of
// channel group g, batch row b, group cg within the row).  x and h_{t-1} are
// staged into `stage` (2 * W * C * 64 elements of T, free on entry) by direct
// loads and read back in the epilogue.  dz_r, dz_i are stored as TZ.  (Used
// by the fused kernel; with z read from memory instead, for the scan entry
// point, the same tile measured 376 against 366 µs for 256 x 2048 x 128 fp32
// and 215-222 against 220-223 µs for 16 x 16384 x 256 bf16, so the scan
// keeps its own kernels.)
// Element offset of one tensor from that of another with a different element
// size (same [B][L][D] index).
template <typename TA, typename TB, typename Off>
__device__ __forceinline__ Off elem_offset(Off off_a) {
    return sizeof(TA) == sizeof(TB) ? off_a : off_a / (Off)sizeof(TA) * (Off)sizeof(TB);
}

template <bool FULL, typename T, typename TH, typename TD, typename TZ, int W, int C, int K,
          typename Off>
__device__ __forceinline__ void bwd_eps_tile(const BwdParams& P, int64_t r, int64_t g, int64_t b,
                                             int64_t cg, const float (&zr)[C],
                                             const float (&zi)[C], char* stage,
                                             Seg (&agg)[W][kWave][1],
                                             uint64_t (&win_sh)[W * K][kWave][1],
                                             float (&carry_sh)[kWave][1],
                                             float (&red)[W][kWave][1], int w, int lane) {
    const int64_t s = P.nseg - 1 - r;  // tile row along L
    const int64_t t0 = s * W * C;
    BwdLane<T, 1, Off> ln;
    ln.init(g, lane, P.L, P.D, P.nch);
    ChannelConst cc[1];
    float h0v[1], dhTv[1];
    bwd_lane_consts<1>(P, ln.c0, ln.d0, cc, h0v, dhTv);
    const int64_t tw = t0 + (int64_t)w * C;
    // FULL: a tile with s > 0 and every step before L (no masks, h_{t-1} of
    // every step from the staged rows); the caller branches on it uniformly.
    constexpr bool full = FULL;
    // x and h_{t-1} are only needed in the epilogue: they wait in LDS, not in
    // registers.
    constexpr int kStaged = C * kWave * (int)sizeof(T);  // one tensor's rows of a wave
    char* const xs = stage + w * 2 * kStaged;
    char* const hs = xs + kStaged;
    static_assert(sizeof(TH) <= sizeof(T), "the staged h rows fit the x rows' room");
    stage_rows<T, C>((const T*)P.x, b, P.L, P.D, cg * kWave, tw, 0, xs, lane);
    stage_rows<TH, C>((const TH*)P.h, b, P.L, P.D, cg * kWave, tw, -1, hs, lane);
    float gv[C];
    // The output gate is folded in only with fp32 x (the gated layer's x');
    // the host passes no gy otherwise.
    if (sizeof(T) == 4 && P.gy) {
        // dh_t = y_t SiLU(z_t) and, with gdz (fp32 h only), dz_t = y_t h_t
        // SiLU'(z_t), SiLU'(v) = s (1 + v (1 - s)), s = sigmoid(v).  h_t is
        // loaded beside dy and hz (the same lines as the staged rows h_{t-1},
        // mostly from the cache); every load is issued before the first store
        // (a store could alias a later load's tensor and would hold it).
        float dzv[C];
        const bool gdz = sizeof(TH) == 4 && P.gdz;
#pragma unroll
        for (int j = 0; j < C; ++j) {
            const int64_t t = tw + j < P.L ? tw + j : P.L - 1;
            const Off off = elem_offset<T, TH>(ln.at(t));
            float y[1], z[1], hv[1] = {0.0f};
            load_vec<TH, 1>((const TH*)P.gy, off, y);
            load_vec<TH, 1>((const TH*)P.gz, off, z);
            if (gdz) load_vec<TH, 1>((const TH*)P.h, off, hv);
            const float sg = sigmoid(z[0]);
            gv[j] = y[0] * (z[0] * sg);
            dzv[j] = y[0] * hv[0] * (sg * fmaf(z[0], 1.0f - sg, 1.0f));
        }
        if (gdz && ln.valid) {
#pragma unroll
            for (int j = 0; j < C; ++j) {
                const float dz[1] = {dzv[j]};
                if (full || tw + j < P.L)
                    store_vec<TH, 1>((TH*)P.gdz, elem_offset<T, TH>(ln.at(tw + j)), dz);
            }
        }
    } else {
#pragma unroll
        for (int j = 0; j < C; ++j) {
            const int64_t t = tw + j < P.L ? tw + j : P.L - 1;
            float v[1];
            load_vec<T, 1>((const T*)P.dh, ln.at(t), v);
            gv[j] = v[0];
        }
    }
    float rr[C], al[C];
#pragma unroll
    for (int j = 0; j < C; ++j) {
        rr[j] = sigmoid(zr[j]);
        al[j] = fast_exp2(rr[j] * cc[0].neg_s_l2);
    }
    {
        Seg sg{1.0f, 0.0f};
#pragma unroll
        for (int j = C - 1; j >= 0; --j) {
            const bool ok = full || tw + j < P.L;
            sg = compose(ok ? Seg{al[j], al[j] * gv[j]} : Seg{1.0f, 0.0f}, sg);
        }
        agg[w][lane][0] = sg;
    }
    __syncthreads();
    // pre: the waves after this one (applied first); tot: the whole tile.
    Seg pre{1.0f, 0.0f}, tot{1.0f, 0.0f};
#pragma unroll
    for (int q = W - 1; q >= 0; --q) {
        const Seg e = agg[q][lane][0];
        if (q > w) pre = compose(e, pre);
        tot = compose(e, tot);
    }
    __syncthreads();  // agg is reused below
    uint64_t* const own = P.lb.states + r * P.nch + ln.c0;
    if (r == 0) {
        if (w == 0) {
            carry_sh[lane][0] = dhTv[0];
            if (ln.valid) publish(own, pack_inclusive(fmaf(tot.A, dhTv[0], tot.H)));
        }
    } else {
        if (w == 0 && ln.valid) publish(own, pack_aggregate(tot));
        lookback_carry<W, 1, K>(P.lb.states, P.nch, ln.c0, r, dhTv, win_sh, carry_sh, w, lane,
                           P.lb.status);
        if (w == 0 && ln.valid)
            publish(own, pack_inclusive(fmaf(tot.A, carry_sh[lane][0], tot.H)));
    }
    __syncthreads();
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): the staged x and h rows are in LDS
    float eps = fmaf(pre.A, carry_sh[lane][0], pre.H);
    float dsum[1] = {0.0f};
#pragma unroll
    for (int j = C - 1; j >= 0; --j) {
        const int64_t t = tw + j;
        if (!(full || t < P.L)) continue;  // past the end: the identity
        const float delta = gv[j] + eps;
        const float rj = rr[j], a = al[j];
        const float i = sigmoid(zi[j]);
        const float mm = one_minus_exp_neg(rj * cc[0].two_s, a);
        const float rs = mm > 0.0f ? fast_rsq(mm) : 0.0f;
        const float sq = mm * rs;  // sqrt(1 - alpha^2)
        const float hprev = !full && t == 0 ? h0v[0] : lds_elem<TH>(hs, j * kWave + lane);
        const float g_alpha = delta * hprev;
        const float gbi = delta * lds_elem<T>(xs, j * kWave + lane) * i;  // dLoss/dbeta * i
        const float gq = fmaf(gbi * (a * a), rs, -a * g_alpha);       // dLoss/dq
        dsum[0] = fmaf(gq, rj, dsum[0]);
        const float dxv[1] = {delta * (sq * i)};
        const float dzrv[1] = {gq * (cc[0].s * fmaf(-rj, rj, rj))};
        const float dziv[1] = {gbi * sq * (1.0f - i)};
        eps = a * delta;
        if (ln.valid) {
            const Off off = ln.at(t);
            store_vec<TD, 1>((TD*)P.dx, z_offset<T, TD>(off), dxv);
            store_vec<TZ, 1>((TZ*)P.dzr, z_offset<T, TZ>(off), dzrv);
            store_vec<TZ, 1>((TZ*)P.dzi, z_offset<T, TZ>(off), dziv);
            if (!full && t == 0 && P.dh0) P.dh0[ln.c0] = eps;
        }
    }
    write_partial<W, 1>(red, dsum, P.partial + s * P.nch + ln.c0, ln.valid, w, lane);
}

// TW: type of the weights and biases (bf16 weights against fp32 x take one
// operand plane).
template <typename T, typename TH, int K, typename Off, typename TW = T>
__global__ __launch_bounds__(fusedz::NT, 4) void
scan_bwd_fused_kernel(BwdParams P, const __bf16* pack, const TW* br, const TW* bi) {
    constexpr int W = fusedz::W, C = fusedz::C;
    // LDS: the tile product, then the x and h staging of the epilogue.
    constexpr size_t kStaging = (size_t)2 * W * C * kWave * sizeof(T);
    constexpr size_t kSmem = fusedz::Tile<T, TW>::kSmem > kStaging
                                 ? fusedz::Tile<T, TW>::kSmem : kStaging;
    __shared__ __attribute__((aligned(16))) char smem[kSmem];
    __shared__ Seg agg[W][kWave][1];
    __shared__ uint64_t win_sh[W * K][kWave][1];
    __shared__ float carry_sh[kWave][1];
    __shared__ float red[W][kWave][1];
    __shared__ int64_t tile_sh;
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int w = wave_id();
    if (tid == 0) tile_sh = (int64_t)atomicAdd(P.lb.ticket, 1u);
    __syncthreads();
    const int64_t tile = tile_sh;
    if (tile >= P.ngroups * P.nseg) return;  // only if the workspace was shared by two calls
    const int64_t r = tile / P.ngroups;  // processing order: from the end of the sequence
    const int64_t g = tile - r * P.ngroups;
    const int64_t s = P.nseg - 1 - r;    // tile row along L
    if (tile == 0) zero_counters(P.dl_counters, P.n_counters);
    const int64_t gpr = P.D / kWave;      // channel groups per batch row
    const int64_t b = g / gpr, cg = g - b * gpr;
    float zr[C], zi[C];
    fusedz::tile_z<T, TW>((const T*)P.x, pack, br, bi, P.L, P.D, b, cg, s * W * C, smem, tid, w,
                          lane, zr, zi);
    __syncthreads();  // every wave holds its z: the product's LDS is free
    if (s > 0 && (s + 1) * W * C <= P.L)
        bwd_eps_tile<true, T, TH, T, float, W, C, K, Off>(P, r, g, b, cg, zr, zi, smem, agg, win_sh,
                                                          carry_sh, red, w, lane);
    else
        bwd_eps_tile<false, T, TH, T, float, W, C, K, Off>(P, r, g, b, cg, zr, zi, smem, agg, win_sh,
                                                           carry_sh, red, w, lane);
}

// ------------------------------------------------------------------ dLambda reduction
// dLambda[d] = sigmoid(Lambda_d) * sum_rows partial[row][d], in double and in a
// fixed order, in one launch: block (nb, dg) sums rows [nb*64, nb*64 + 64) of
// channels [dg*64, dg*64 + 64) into partial2[nb]; the last block of column
// group dg to finish (a counter per group, zeroed by the scan kernel that
// wrote the partials) adds the row-block sums in a fixed order, so the result
// does not depend on which block finishes last.
__global__ __launch_bounds__(256) void dlambda_kernel(const float* __restrict__ partial,
                                                      double* __restrict__ partial2,
                                                      int64_t rows, int64_t D,
                                                      const float* __restrict__ lam,
                                                      float* __restrict__ dlambda,
                                                      unsigned* __restrict__ counters) {
    __shared__ double red[4][kWave];
    __shared__ int last_sh;
    const int lane = threadIdx.x & (kWave - 1);
    const int w = threadIdx.x / kWave;
    const int64_t d = (int64_t)blockIdx.y * kWave + lane;
    const int64_t nb = blockIdx.x;
    double acc = 0.0;
    if (d < D) {
        // All loads first (rows past the end read the last row and count as
        // zero), then the sum in row order.
        const int64_t r0 = nb * kReduceRows + w * (kReduceRows / 4);
        float v[kReduceRows / 4];
#pragma unroll
        for (int k = 0; k < kReduceRows / 4; ++k) {
            const int64_t row = r0 + k < rows ? r0 + k : rows - 1;
            v[k] = partial[row * D + d];
        }
#pragma unroll
        for (int k = 0; k < kReduceRows / 4; ++k)
            if (r0 + k < rows) acc += (double)v[k];
    }
    red[w][lane] = acc;
    __syncthreads();
    // partial2 and the counter travel as agent-scope atomics, which this GPU
    // keeps coherent across its L2s (as the look-back state words): each
    // block's sums are complete in memory (vmcnt(0)) before its counter
    // increment is issued, and the last block reads them back with atomic
    // loads.  No release fence, which would write back the whole L2.
    if (w == 0 && d < D) {
        const double v = ((red[0][lane] + red[1][lane]) + red[2][lane]) + red[3][lane];
        __hip_atomic_store((uint64_t*)(partial2 + nb * D + d), __builtin_bit_cast(uint64_t, v),
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0)
        last_sh = __hip_atomic_fetch_add(counters + blockIdx.y, 1u, __ATOMIC_RELAXED,
                                         __HIP_MEMORY_SCOPE_AGENT) == gridDim.x - 1;
    __syncthreads();
    if (!last_sh) return;
    // Wave w sums its contiguous run of row blocks in ascending order; the
    // four runs are then added in order.
    const int64_t nblk = gridDim.x;
    const int64_t per = (nblk + 3) / 4;
    const int64_t k0 = w * per, k1 = k0 + per < nblk ? k0 + per : nblk;
    double s = 0.0;
    if (d < D) {
#pragma unroll 8
        for (int64_t k = k0; k < k1; ++k)
            s += __builtin_bit_cast(double, __hip_atomic_load((uint64_t*)(partial2 + k * D + d),
                                                              __ATOMIC_RELAXED,
                                                              __HIP_MEMORY_SCOPE_AGENT));
    }
    __syncthreads();  // red is reused
    red[w][lane] = s;
    __syncthreads();
    if (w != 0 || d >= D) return;
    const double t = ((red[0][lane] + red[1][lane]) + red[2][lane]) + red[3][lane];
    const double lv = (double)lam[d];
    dlambda[d] = (float)(t / (1.0 + exp(-lv)));
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

// ------------------------------------------------------------------ launch plan
// Tile shapes: W waves per workgroup and E elements per lane per macro-chunk
// (C = E / VEC steps per wave), so a wave moves the same bytes per
// macro-chunk whatever VEC is.
// The chain kernel runs 8 waves of 4 or 5 steps (macro-chunks of 32 or 40
// steps), whichever pads L less: 2048 x 200 x 64 fp32 backward 151 us with 40
// (200 = 5 x 40), against 158 us with 32 and 168-173 us with 16 waves of 4
// (64 steps: 200 = 3 x 64 + 8, the last macro-chunk one eighth used).
#ifndef RECBLR_BWD_CHAIN_W
#define RECBLR_BWD_CHAIN_W 8
#endif
#ifndef RECBLR_BWD_LB_W
#define RECBLR_BWD_LB_W 8
#endif
#ifndef RECBLR_BWD_LB_E
#define RECBLR_BWD_LB_E 16
#endif
// Channels per lane at most, per kernel (measured best on MI355X).
#ifndef RECBLR_BWD_CHAIN_MAX_VEC
#define RECBLR_BWD_CHAIN_MAX_VEC 1
#endif
#ifndef RECBLR_BWD_LB_MAX_VEC
#define RECBLR_BWD_LB_MAX_VEC 1
#endif
constexpr int kChainW = RECBLR_BWD_CHAIN_W;
// Steps per wave of the chain kernel for a sequence of L steps.
inline int chain_steps(int64_t L) {
    const int64_t p4 = (L + 4 * kChainW - 1) / (4 * kChainW) * (4 * kChainW);
    const int64_t p5 = (L + 5 * kChainW - 1) / (5 * kChainW) * (5 * kChainW);
    return p5 < p4 ? 5 : 4;
}
// bf16 I/O takes 12 steps per wave: with the step pairs formed on use that is
// 126 VGPRs, two workgroups per compute unit (16 x 16384 x 256 backward:
// 222 us against 255 us at 16 steps); fp32 I/O keeps 16 (256 x 2048 x 128:
// 370 us against 410 us at 12).
#ifndef RECBLR_BWD_LB_E_BF16
#define RECBLR_BWD_LB_E_BF16 12
#endif
constexpr int kLbW = RECBLR_BWD_LB_W;
constexpr int lb_elems(size_t esz) { return esz == 2 ? RECBLR_BWD_LB_E_BF16 : RECBLR_BWD_LB_E; }
// Look-back window per wave: K tiles, K * VEC state words per lane.
#ifndef RECBLR_BWD_LB_WORDS
#define RECBLR_BWD_LB_WORDS 1
#endif
template <int VEC>
constexpr int lb_window() { return RECBLR_BWD_LB_WORDS / VEC > 0 ? RECBLR_BWD_LB_WORDS / VEC : 1; }
template <int E, int VEC>
constexpr int steps_per_wave() { return E / VEC > 0 ? E / VEC : 1; }
// Steps of one look-back tile for a given VEC.
constexpr int64_t lb_tile_steps(size_t esz, int vec) {
    return (int64_t)kLbW * (lb_elems(esz) / vec > 0 ? lb_elems(esz) / vec : 1);
}
// Lanes of the chain kernel take as many channels as keep this many
// workgroups (one per compute unit).
constexpr int64_t kChainMinGroups = 256;
// The chain kernel runs when it has at least four workgroups per compute
// unit; below that the look-back kernel is faster (its 16 steps per wave
// amortise the carry fold over four times as many steps as the chain
// kernel's 4; 256 x 2048 x 128 fp32: 378 us against 404 us on MI355X),
// above it the chain kernel is (2048 x 200 x 64: 177 us against 183 us).
#ifndef RECBLR_BWD_LB_BELOW
#define RECBLR_BWD_LB_BELOW 1024
#endif
constexpr int64_t kLookbackBelowGroups = RECBLR_BWD_LB_BELOW;
// Largest channels-per-lane of a kernel for an element size (8-byte accesses
// per lane at most).
constexpr int max_vec(size_t esz, bool lookback, int64_t nch = INT64_MAX) {
    const int cap = lookback ? RECBLR_BWD_LB_MAX_VEC : RECBLR_BWD_CHAIN_MAX_VEC;
    int v = (int)(8 / esz) < cap ? (int)(8 / esz) : cap;
    while (v > 1 && !lookback && nch / (kWave * v) < kChainMinGroups) v /= 2;
    return v;
}

struct BwdPlan {
    bool lookback;
    int vec;
    int64_t ngroups, nseg;
};

// The mode depends only on (B, L, D); the tile count also on VEC (see the
// forward launcher).
static bool backward_uses_lookback(int64_t B, int64_t L, int64_t D, size_t esz) {
    const int64_t groups_one = (B * D + kWave - 1) / kWave;
    return groups_one < kLookbackBelowGroups && L > lb_tile_steps(esz, max_vec(esz, true));
}

static BwdPlan plan_backward(int64_t B, int64_t L, int64_t D, size_t esz, int vec) {
    BwdPlan p;
    p.vec = vec;
    p.lookback = backward_uses_lookback(B, L, D, esz);
    p.ngroups = (B * D / vec + kWave - 1) / kWave;
    p.nseg = p.lookback ? (L + lb_tile_steps(esz, vec) - 1) / lb_tile_steps(esz, vec) : 1;
    return p;
}

static int pick_vec_bwd(const ScanBwdArgs& a) {
    const size_t esz = io_bytes(a.io), zsz = io_bytes(a.zio);
    const uintptr_t xm = (uintptr_t)a.x | (uintptr_t)a.h | (uintptr_t)a.dh | (uintptr_t)a.dx;
    const uintptr_t zm = (uintptr_t)a.zr | (uintptr_t)a.zi | (uintptr_t)a.dzr | (uintptr_t)a.dzi;
    const uintptr_t sm = (uintptr_t)a.h0 | (uintptr_t)a.dhT | (uintptr_t)a.dh0;
    for (int v = max_vec(esz, backward_uses_lookback(a.B, a.L, a.D, esz), a.B * a.D); v > 1;
         v /= 2)
        if (a.D % v == 0 && xm % (v * esz) == 0 && zm % (v * zsz) == 0 && sm % (v * 4) == 0)
            return v;
    return 1;
}

// Workspace: [look-back states][dLambda partials (nseg rows of B*D)][row-block sums].
struct BwdLayout {
    size_t lb, partial, partial2, counters, total;
};

inline int64_t dlambda_groups(int64_t D) { return (D + kWave - 1) / kWave; }

static BwdLayout bwd_layout(int64_t B, int64_t D, const BwdPlan& p) {
    BwdLayout l;
    const int64_t rows = p.nseg * B;
    const int64_t nb = (rows + kReduceRows - 1) / kReduceRows;
    l.lb = 0;  // the header (ticket, status word) is there in both modes
    l.partial = align_up(p.lookback ? lookback_ws_bytes(p.nseg, B * D) : 256);
    l.partial2 = l.partial + align_up((size_t)(rows * D) * sizeof(float));
    l.counters = l.partial2 + align_up((size_t)(nb * D) * sizeof(double));
    l.total = l.counters + align_up((size_t)dlambda_groups(D) * sizeof(unsigned));
    return l;
}

size_t scan_backward_workspace(int64_t B, int64_t L, int64_t D, IoType io) {
    const size_t esz = io_bytes(io);
    const bool lb = backward_uses_lookback(B, L, D, esz);
    return bwd_layout(B, D, plan_backward(B, L, D, esz, max_vec(esz, lb))).total;
}

// ev0 / ev1 (may be null) take the scan kernel's start and end times.
template <typename TX, typename TZ, typename Off, int VEC>
static hipError_t launch_bwd_vec(const BwdParams& P, const BwdPlan& plan, hipStream_t stream,
                                 hipEvent_t ev0, hipEvent_t ev1) {
    if (!plan.lookback) {
        // The chain kernel takes one channel per lane (RECBLR_BWD_CHAIN_MAX_VEC).
        if constexpr (VEC != 1) {
            return hipErrorInvalidValue;
        } else {
            const dim3 grid((unsigned)plan.ngroups), block(kChainW * kWave);
            if (chain_steps(P.L) == 5)
                return launch_measured(scan_bwd_chain_kernel<TX, TZ, kChainW, 5, 1, Off>, grid,
                                       block, stream, ev0, ev1, P);
            return launch_measured(scan_bwd_chain_kernel<TX, TZ, kChainW, 4, 1, Off>, grid, block,
                                   stream, ev0, ev1, P);
        }
    }
    hipError_t e = lookback_reset(P.lb, plan.nseg * P.nch, stream);
    if (e != hipSuccess) return e;
    const dim3 grid((unsigned)(plan.ngroups * plan.nseg)), block(kLbW * kWave);
    return launch_measured(scan_bwd_lookback_kernel<TX, TZ, kLbW,
                                                    steps_per_wave<lb_elems(sizeof(TX)), VEC>(),
                                                    VEC, lb_window<VEC>(), Off>,
                           grid, block, stream, ev0, ev1, P);
}

template <typename TX, typename TZ>
static hipError_t launch_bwd_typed(const BwdParams& P, const BwdPlan& plan, hipStream_t stream,
                                   hipEvent_t ev0, hipEvent_t ev1) {
    // 32-bit byte offsets whenever a whole [B, L, D] tensor spans less than 4 GiB.
    const bool small = (uint64_t)(P.nch * P.L) * sizeof(TZ) < (1ull << 32);
    // VEC = 4 only exists for 2-byte x (8-byte accesses per lane).
    if (small) {
        if constexpr (sizeof(TX) == 2)
            if (plan.vec == 4) return launch_bwd_vec<TX, TZ, uint32_t, 4>(P, plan, stream, ev0, ev1);
        if (plan.vec == 2) return launch_bwd_vec<TX, TZ, uint32_t, 2>(P, plan, stream, ev0, ev1);
        return launch_bwd_vec<TX, TZ, uint32_t, 1>(P, plan, stream, ev0, ev1);
    }
    if constexpr (sizeof(TX) == 2)
        if (plan.vec == 4) return launch_bwd_vec<TX, TZ, uint64_t, 4>(P, plan, stream, ev0, ev1);
    if (plan.vec == 2) return launch_bwd_vec<TX, TZ, uint64_t, 2>(P, plan, stream, ev0, ev1);
    return launch_bwd_vec<TX, TZ, uint64_t, 1>(P, plan, stream, ev0, ev1);
}

// dLambda from the per-tile partials [rows][D]: one fixed-order launch.
static hipError_t launch_dlambda(const float* partial, double* partial2, int64_t rows, int64_t D,
                                 const float* lambda, float* dlambda, unsigned* counters,
                                 hipStream_t stream) {
    const int64_t nblk = (rows + kReduceRows - 1) / kReduceRows;
    dim3 grid((unsigned)nblk, (unsigned)dlambda_groups(D));
    hipLaunchKernelGGL(dlambda_kernel, grid, dim3(256), 0, stream, partial, partial2, rows, D,
                       lambda, dlambda, counters);
    return hipGetLastError();
}

hipError_t launch_scan_backward(const ScanBwdArgs& a, hipStream_t stream) {
    const BwdPlan plan = plan_backward(a.B, a.L, a.D, io_bytes(a.io), pick_vec_bwd(a));
    const BwdLayout lay = bwd_layout(a.B, a.D, plan);
    char* ws = (char*)a.ws;
    float* partial = (float*)(ws + lay.partial);
    double* partial2 = (double*)(ws + lay.partial2);
    unsigned* counters = (unsigned*)(ws + lay.counters);
    const BwdParams P{a.x,   a.zr,    a.zi,  a.lambda, a.h0, a.h,   a.dh,  a.dhT,
                      a.dx,  a.dzr,   a.dzi, a.dh0,    partial, a.L, a.D,  a.B * a.D,
                      plan.ngroups, plan.nseg,
                      plan.lookback ? lookback_ws(ws + lay.lb)
                                    : LookbackWs{nullptr, lookback_ws(ws + lay.lb).status, nullptr},
                      counters, dlambda_groups(a.D)};
    hipError_t e;
    if (a.io == IoType::kF32)
        e = launch_bwd_typed<float, float>(P, plan, stream, a.ev_begin, a.ev_end);
    else if (a.zio == IoType::kF32)
        e = launch_bwd_typed<bf16, float>(P, plan, stream, a.ev_begin, a.ev_end);
    else e = launch_bwd_typed<bf16, bf16>(P, plan, stream, a.ev_begin, a.ev_end);
    if (e != hipSuccess) return e;
    return launch_dlambda(partial, partial2, plan.nseg * a.B, a.D, a.lambda, a.dlambda, counters,
                          stream);
}

// ------------------------------------------------------------------ fused backward
static BwdPlan plan_fused_backward(int64_t B, int64_t L, int64_t D) {
    constexpr int64_t kSteps = (int64_t)fusedz::W * fusedz::C;
    BwdPlan p;
    p.lookback = true;
    p.vec = 1;
    p.ngroups = (B * D + kWave - 1) / kWave;
    p.nseg = (L + kSteps - 1) / kSteps;
    return p;
}

bool fused_backward_applies(int64_t B, int64_t L, int64_t D, IoType io, const void* x,
                            const void* h, const void* pack) {
    const size_t esz = io_bytes(io);
    // x and h are staged with 16-byte direct-to-LDS loads (stage_rows): both
    // must start on a 16-byte boundary, as must the packed weights.
    return B > 0 && L > 0 && D > 0 && D % kWave == 0 &&
           ((uintptr_t)x | (uintptr_t)h | (uintptr_t)pack) % 16 == 0 &&
           (L + fastmm::BM) * D * (int64_t)esz < ((int64_t)1 << 31);
}

size_t fused_backward_workspace(int64_t B, int64_t L, int64_t D) {
    if (B <= 0 || L <= 0 || D <= 0) return 0;
    return bwd_layout(B, D, plan_fused_backward(B, L, D)).total;
}

hipError_t launch_fused_backward(const FusedBwdArgs& a, hipStream_t stream) {
    // the output gate is folded into the fp32-x kernels only
    if (a.gy && io_bytes(a.io) != 4) return hipErrorInvalidValue;
    const BwdPlan plan = plan_fused_backward(a.B, a.L, a.D);
    const BwdLayout lay = bwd_layout(a.B, a.D, plan);
    char* ws = (char*)a.ws;
    float* partial = (float*)(ws + lay.partial);
    double* partial2 = (double*)(ws + lay.partial2);
    unsigned* counters = (unsigned*)(ws + lay.counters);
    const BwdParams P{a.x,  nullptr, nullptr, a.lambda, a.h0, a.h,   a.dh,  a.dhT,
                      a.dx, a.dzr,   a.dzi,   a.dh0,    partial, a.L, a.D,  a.B * a.D,
                      plan.ngroups, plan.nseg, lookback_ws(ws + lay.lb),
                      counters, dlambda_groups(a.D), a.gy, a.gz, a.gdz};
    hipError_t e = lookback_reset(P.lb, plan.nseg * P.nch, stream);
    if (e != hipSuccess) return e;
    const dim3 grid((unsigned)(plan.ngroups * plan.nseg)), block(fusedz::NT);
    const size_t esz = io_bytes(a.io);
    const bool small = (uint64_t)(a.B * a.L * a.D) * 4 < (1ull << 32);
    constexpr int K = lb_window<1>();
    if (esz == 4 && !a.h_bf16) {
        if (small)
            hipLaunchKernelGGL((scan_bwd_fused_kernel<float, float, K, uint32_t>), grid, block, 0,
                               stream, P, (const __bf16*)a.pack, (const float*)a.br,
                               (const float*)a.bi);
        else
            hipLaunchKernelGGL((scan_bwd_fused_kernel<float, float, K, uint64_t>), grid, block, 0,
                               stream, P, (const __bf16*)a.pack, (const float*)a.br,
                               (const float*)a.bi);
    } else if (a.h_bf16) {
        // fp32 x; h, the weights (one packed plane) and biases in bf16
        if (small)
            hipLaunchKernelGGL((scan_bwd_fused_kernel<float, bf16, K, uint32_t, bf16>), grid,
                               block, 0, stream, P, (const __bf16*)a.pack, (const bf16*)a.br,
                               (const bf16*)a.bi);
        else
            hipLaunchKernelGGL((scan_bwd_fused_kernel<float, bf16, K, uint64_t, bf16>), grid,
                               block, 0, stream, P, (const __bf16*)a.pack, (const bf16*)a.br,
                               (const bf16*)a.bi);
    } else {
        if (small)
            hipLaunchKernelGGL((scan_bwd_fused_kernel<bf16, bf16, K, uint32_t>), grid, block, 0,
                               stream, P, (const __bf16*)a.pack, (const bf16*)a.br,
                               (const bf16*)a.bi);
        else
            hipLaunchKernelGGL((scan_bwd_fused_kernel<bf16, bf16, K, uint64_t>), grid, block, 0,
                               stream, P, (const __bf16*)a.pack, (const bf16*)a.br,
                               (const bf16*)a.bi);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return launch_dlambda(partial, partial2, plan.nseg * a.B, a.D, a.lambda, a.dlambda, counters,
                          stream);
}

}  // namespace recblr
