// Forward BD-LRU scan for gfx950: gate activation fused into the load,
// chunked along the sequence, carries combined through LDS and, for long
// sequences over few channels, across workgroups by decoupled look-back.
//
// Recurrence (RecBLR, arXiv 2406.12580, eq:linrnn):  h_t = alpha_t h_{t-1} + beta'_t,
// beta'_t = beta_t x_t, with alpha, beta from the gate equations of section 3.2.
// The parallel form follows section 3.3: every segment of steps is an (A, H)
// pair, pairs compose with the associative operator "bullet", and the state at
// any step is the composition of all earlier segments applied to h0.
//
// Work decomposition:
//   * a lane owns VEC consecutive channels (b, d..d+VEC-1); the 64 lanes of a
//     wave own 64*VEC consecutive flattened channels c = b*D + d, so the loads
//     and stores of one time step are one contiguous run of 64*VEC elements;
//   * a workgroup of W waves owns one channel group; its macro-chunk of W*C
//     steps is split so that wave w scans steps [w*C, w*C + C) sequentially
//     in registers and publishes its aggregate (A, H) in LDS;
//   * chain kernel: the workgroup walks the whole sequence, macro-chunk after
//     macro-chunk, keeping the carry in registers and the next macro-chunk's
//     loads in flight (register double buffer);
//   * look-back kernel: every workgroup takes one (group, macro-chunk) tile in
//     ticket order, publishes the tile aggregate, reads the state words of the
//     preceding tiles (each wave a window of K of them, in parallel) and
//     publishes its inclusive state (lookback.hpp).
// Each input element is read once and each output element written once.
#include "device_common.hpp"
#include "launch.hpp"
#include "lookback.hpp"
#include "fused_z.hpp"
#include "mfma_tile.hpp"

namespace recblr {

struct FwdParams {
    const void* p0;  // gated: x;    raw: a
    const void* p1;  // gated: z_r;  raw: u
    const void* p2;  // gated: z_i
    const float* lam;
    const float* h0;
    void* h;
    float* hT;
    int64_t L, D, nch;      // nch = B * D
    int64_t ngroups, nseg;  // channel groups; tiles along L (look-back kernel)
    LookbackWs lb;
};

// One lane's channels and addressing.
template <typename TX, int VEC, typename Off>
struct LaneChannels {
    bool valid;
    int64_t c0;  // first channel (valid lanes) or 0 (idle lanes shadow channel 0)
    int64_t d0;
    Off base;    // byte offset of (b, 0, d) in an x-typed tensor
    Off row;     // bytes between consecutive time steps

    __device__ __forceinline__ void init(int64_t group, int lane, int64_t L, int64_t D,
                                         int64_t nch) {
        const int64_t c = (group * kWave + lane) * VEC;
        valid = c < nch;
        c0 = valid ? c : 0;
        const int64_t b = c0 / D;
        d0 = c0 - b * D;
        base = (Off)((b * L * D + d0) * (int64_t)sizeof(TX));
        row = (Off)(D * (int64_t)sizeof(TX));
    }
    __device__ __forceinline__ Off at(int64_t t) const { return base + (Off)t * row; }
};

// Raw inputs of C steps; steps past the end re-read step L-1 (in bounds) and
// are masked when the gates are formed.
template <typename TX, typename TZ, int C, int VEC, bool RAW, typename Off>
struct ChunkIn {
    float v0[C][VEC], v1[C][VEC], v2[C][VEC];

    // FULL: every step is before L (no clamping needed).
    template <bool FULL>
    __device__ __forceinline__ void fetch(const FwdParams& P, const LaneChannels<TX, VEC, Off>& ln,
                                          int64_t t_first) {
#pragma unroll
        for (int j = 0; j < C; ++j) {
            const int64_t t = FULL || t_first + j < P.L ? t_first + j : P.L - 1;
            const Off off = ln.at(t);
            load_vec<TX, VEC>((const TX*)P.p0, off, v0[j]);
            load_vec<TZ, VEC>((const TZ*)P.p1, z_offset<TX, TZ>(off), v1[j]);
            if (!RAW) load_vec<TZ, VEC>((const TZ*)P.p2, z_offset<TX, TZ>(off), v2[j]);
        }
    }
};

// (alpha_t, beta'_t) of C steps from the raw inputs; masked steps are the
// identity (1, 0).  FULL: no step is masked.
template <bool FULL, typename TX, typename TZ, int C, int VEC, bool RAW, typename Off>
__device__ __forceinline__ void form_steps(const ChunkIn<TX, TZ, C, VEC, RAW, Off>& in,
                                           const ChannelConst (&cc)[VEC], int64_t t_first,
                                           int64_t L, float (&a)[C][VEC], float (&u)[C][VEC]) {
#pragma unroll
    for (int j = 0; j < C; ++j) {
        const bool ok = FULL || t_first + j < L;
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
            float aj, uj;
            if (RAW) {
                aj = in.v0[j][k];
                uj = in.v1[j][k];
            } else {
                gate_forward<sizeof(TX) == 4>(in.v0[j][k], in.v1[j][k], in.v2[j][k], cc[k], aj,
                                              uj);
            }
            a[j][k] = ok ? aj : 1.0f;
            u[j][k] = ok ? uj : 0.0f;
        }
    }
}

// Run C steps on from the states hv and store h (steps before L only).
template <bool FULL, typename TX, int C, int VEC, typename Off>
__device__ __forceinline__ void emit_steps(const FwdParams& P, const LaneChannels<TX, VEC, Off>& ln,
                                           int64_t t_first, const float (&a)[C][VEC],
                                           const float (&u)[C][VEC], float (&hv)[VEC]) {
#pragma unroll
    for (int j = 0; j < C; ++j) {
#pragma unroll
        for (int k = 0; k < VEC; ++k) hv[k] = fmaf(a[j][k], hv[k], u[j][k]);
        if (ln.valid && (FULL || t_first + j < P.L))
            store_vec<TX, VEC>((TX*)P.h, ln.at(t_first + j), hv);
    }
}

template <int VEC>
__device__ __forceinline__ void load_consts(const float* lam, int64_t d0,
                                            ChannelConst (&cc)[VEC]) {
#pragma unroll
    for (int k = 0; k < VEC; ++k) cc[k] = channel_const(lam[d0 + k]);
}

// ------------------------------------------------------------------ chain kernel
// One macro-chunk: gates, local aggregates through LDS, carry fold, store.
template <bool FULL, typename TX, typename TZ, int W, int C, int VEC, bool RAW, typename Off>
__device__ __forceinline__ void chain_fwd_step(const FwdParams& P,
                                               const LaneChannels<TX, VEC, Off>& ln,
                                               const ChunkIn<TX, TZ, C, VEC, RAW, Off>& cur,
                                               const ChannelConst (&cc)[VEC],
                                               Seg (&agg)[W][kWave][VEC], int64_t tw, int w,
                                               int lane, float (&carry)[VEC]) {
    float a[C][VEC], u[C][VEC];
    form_steps<FULL>(cur, cc, tw, P.L, a, u);
#pragma unroll
    for (int k = 0; k < VEC; ++k) {
        Seg s{1.0f, 0.0f};
#pragma unroll
        for (int j = 0; j < C; ++j) s = compose(Seg{a[j][k], u[j][k]}, s);
        agg[w][lane][k] = s;
    }
    __syncthreads();
    // Carry into this wave: fold the earlier waves' aggregates onto the carry.
    float hv[VEC], cout[VEC];
#pragma unroll
    for (int k = 0; k < VEC; ++k) hv[k] = carry[k];
#pragma unroll
    for (int q = 0; q < W; ++q) {
        if (q < w) {
#pragma unroll
            for (int k = 0; k < VEC; ++k) {
                const Seg e = agg[q][lane][k];
                hv[k] = fmaf(e.A, hv[k], e.H);
            }
        }
    }
#pragma unroll
    for (int k = 0; k < VEC; ++k) cout[k] = hv[k];
    emit_steps<FULL, TX, C, VEC, Off>(P, ln, tw, a, u, hv);
    // Carry out of the macro-chunk: the fold continued through the last wave.
#pragma unroll
    for (int q = 0; q < W; ++q) {
        if (q >= w) {
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

// The steady-state loop covers the full macro-chunks and has no branch
// around a memory instruction: on this GPU loads and stores share one
// in-order counter, and a branch that issues a different number of them
// makes the compiler wait for every outstanding load, including the
// prefetched next chunk.  The next chunk's loads are always issued (clamped
// to step L-1 past the end); a partial last macro-chunk runs after the loop.
template <typename TX, typename TZ, int W, int C, int VEC, bool RAW, typename Off>
__global__ __launch_bounds__(W* kWave) void scan_fwd_chain_kernel(FwdParams P) {
    __shared__ Seg agg[2][W][kWave][VEC];
    const int lane = threadIdx.x & (kWave - 1);
    const int w = wave_id();
    LaneChannels<TX, VEC, Off> ln;
    ln.init(blockIdx.x, lane, P.L, P.D, P.nch);
    ChannelConst cc[VEC];
    if (!RAW) load_consts<VEC>(P.lam, ln.d0, cc);
    float carry[VEC];
#pragma unroll
    for (int k = 0; k < VEC; ++k) carry[k] = P.h0 ? P.h0[ln.c0 + k] : 0.0f;

    constexpr int64_t kMacro = (int64_t)W * C;
    const int64_t nfull = P.L / kMacro;
    const bool tail = nfull * kMacro < P.L;
    // Two buffers alternate roles (loop unrolled by two), so no register copy
    // ties the prefetched chunk to the one being consumed.
    ChunkIn<TX, TZ, C, VEC, RAW, Off> bufA, bufB;
    const int64_t woff = (int64_t)w * C;
    if (P.L > 0) bufA.template fetch<false>(P, ln, woff);
    for (int64_t m = 0;;) {
        if (m >= nfull) {
            if (tail) chain_fwd_step<false>(P, ln, bufA, cc, agg[m & 1], m * kMacro + woff, w, lane, carry);
            break;
        }
        bufB.template fetch<false>(P, ln, (m + 1) * kMacro + woff);
        chain_fwd_step<true>(P, ln, bufA, cc, agg[m & 1], m * kMacro + woff, w, lane, carry);
        ++m;
        if (m >= nfull) {
            if (tail) chain_fwd_step<false>(P, ln, bufB, cc, agg[m & 1], m * kMacro + woff, w, lane, carry);
            break;
        }
        bufA.template fetch<false>(P, ln, (m + 1) * kMacro + woff);
        chain_fwd_step<true>(P, ln, bufB, cc, agg[m & 1], m * kMacro + woff, w, lane, carry);
        ++m;
    }
    if (w == 0 && ln.valid && P.hT) {
#pragma unroll
        for (int k = 0; k < VEC; ++k) P.hT[ln.c0 + k] = carry[k];
    }
}

// ------------------------------------------------------------------ look-back kernel
template <typename TX, typename TZ, int W, int C, int VEC, int K, typename Off>
__global__ __launch_bounds__(W* kWave) void scan_fwd_lookback_kernel(FwdParams P) {
    __shared__ Seg agg[W][kWave][VEC];
    __shared__ uint64_t win_sh[W * K][kWave][VEC];
    __shared__ float carry_sh[kWave][VEC];
    __shared__ int64_t tile_sh;
    const int lane = threadIdx.x & (kWave - 1);
    const int w = wave_id();
    if (threadIdx.x == 0) tile_sh = (int64_t)atomicAdd(P.lb.ticket, 1u);
    __syncthreads();
    const int64_t tile = tile_sh;
    if (tile >= P.ngroups * P.nseg) return;  // only if the workspace was shared by two calls
    const int64_t s = tile / P.ngroups;  // tiles are handed out one tile-row at a time
    const int64_t g = tile - s * P.ngroups;

    LaneChannels<TX, VEC, Off> ln;
    ln.init(g, lane, P.L, P.D, P.nch);
    ChannelConst cc[VEC];
    load_consts<VEC>(P.lam, ln.d0, cc);
    float h0v[VEC];
#pragma unroll
    for (int k = 0; k < VEC; ++k) h0v[k] = P.h0 ? P.h0[ln.c0 + k] : 0.0f;

    const int64_t tw = s * W * C + (int64_t)w * C;
    const bool full = (s + 1) * W * C <= P.L;  // workgroup-uniform
    float a[C][VEC], u[C][VEC];
    {
        ChunkIn<TX, TZ, C, VEC, false, Off> in;
        if (full) {
            in.template fetch<true>(P, ln, tw);
            form_steps<true>(in, cc, tw, P.L, a, u);
        } else {
            in.template fetch<false>(P, ln, tw);
            form_steps<false>(in, cc, tw, P.L, a, u);
        }
    }
#pragma unroll
    for (int k = 0; k < VEC; ++k) {
        Seg sg{1.0f, 0.0f};
#pragma unroll
        for (int j = 0; j < C; ++j) sg = compose(Seg{a[j][k], u[j][k]}, sg);
        agg[w][lane][k] = sg;
    }
    __syncthreads();
    // pre: the waves before this one; tot: the whole tile.
    Seg pre[VEC], tot[VEC];
#pragma unroll
    for (int k = 0; k < VEC; ++k) pre[k] = tot[k] = Seg{1.0f, 0.0f};
#pragma unroll
    for (int q = 0; q < W; ++q) {
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
            const Seg e = agg[q][lane][k];
            if (q < w) pre[k] = compose(e, pre[k]);
            tot[k] = compose(e, tot[k]);
        }
    }
    __syncthreads();  // agg is reused below

    uint64_t* const own = P.lb.states + s * P.nch + ln.c0;
    if (s == 0) {
        if (w == 0) {
#pragma unroll
            for (int k = 0; k < VEC; ++k) {
                carry_sh[lane][k] = h0v[k];
                if (ln.valid) publish(own + k, pack_inclusive(fmaf(tot[k].A, h0v[k], tot[k].H)));
            }
        }
    } else {
        if (w == 0 && ln.valid) {
#pragma unroll
            for (int k = 0; k < VEC; ++k) publish(own + k, pack_aggregate(tot[k]));
        }
        lookback_carry<W, VEC, K>(P.lb.states, P.nch, ln.c0, s, h0v, win_sh, carry_sh, w, lane,
                           P.lb.status);
        if (w == 0 && ln.valid) {
#pragma unroll
            for (int k = 0; k < VEC; ++k)
                publish(own + k, pack_inclusive(fmaf(tot[k].A, carry_sh[lane][k], tot[k].H)));
        }
    }
    __syncthreads();
    float hv[VEC];
#pragma unroll
    for (int k = 0; k < VEC; ++k) hv[k] = fmaf(pre[k].A, carry_sh[lane][k], pre[k].H);
    if (full) emit_steps<true, TX, C, VEC, Off>(P, ln, tw, a, u, hv);
    else emit_steps<false, TX, C, VEC, Off>(P, ln, tw, a, u, hv);
    if (s == P.nseg - 1 && w == W - 1 && ln.valid && P.hT) {
#pragma unroll
        for (int k = 0; k < VEC; ++k) P.hT[ln.c0 + k] = hv[k];
    }
}

// ------------------------------------------------------------------ projections fused in
// Look-back kernel that computes its own gate pre-activations (fused_z.hpp):
// the tile's z for 128 steps x 64 channels (both gates) is one 128 x 128
// matrix-core product, each wave receives its 16 steps in the lane-per-channel
// layout, and the scan proceeds as in the look-back kernel.  z never reaches
// HBM: the kernel reads x and writes h.
namespace fusedfwd {
// Gated-layer output (the output gate of Algorithm alg:gated_recurrent): with GATED the
// kernel stores y = h * SiLU(hz) (and h only where asked for).
struct GatedArgs {
    const void* hz;  // [B][L][D], I/O type
    void* y;         // [B][L][D], I/O type
};

__device__ __forceinline__ float silu(float c) { return c * sigmoid(c); }
}  // namespace fusedfwd

// P.p0 is x; P.p1, P.p2 are unused; P.h may be null for GATED (then only y
// is stored).  pack: [W_r; W_i] ordered by channel
// group of 64 (launch_pack_groups); D % 64 == 0.
// Occupancy: 3 workgroups per CU for bf16 I/O (LDS 48 KB each, 6 waves per
// SIMD), 2 for fp32 (its split operands double the staging LDS).
template <typename T, int K, typename Off, bool GATED>
__global__ __launch_bounds__(fusedz::NT, sizeof(T) == 2 ? 6 : 4) void
scan_fwd_fused_kernel(FwdParams P, const __bf16* pack, const T* br, const T* bi,
                      fusedfwd::GatedArgs G) {
    constexpr int W = fusedz::W, C = fusedz::C;
    __shared__ __attribute__((aligned(16))) char smem[fusedz::Tile<T>::kSmem];
    __shared__ Seg agg[W][kWave][1];
    __shared__ uint64_t win_sh[W * K][kWave][1];
    __shared__ float carry_sh[kWave][1];
    __shared__ int64_t tile_sh;
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int w = wave_id();
    if (tid == 0) tile_sh = (int64_t)atomicAdd(P.lb.ticket, 1u);
    __syncthreads();
    const int64_t tile = tile_sh;
    if (tile >= P.ngroups * P.nseg) return;  // only if the workspace was shared by two calls
    const int64_t s = tile / P.ngroups;
    const int64_t g = tile - s * P.ngroups;
    const int64_t gpr = P.D / kWave;  // channel groups per batch row
    const int64_t b = g / gpr, cg = g - b * gpr;
    const int64_t t0 = s * W * C;
    float zr[C], zi[C];
    fusedz::tile_z<T>((const T*)P.p0, pack, br, bi, P.L, P.D, b, cg, t0, smem, tid, w, lane, zr,
                      zi);

    // ---- the look-back scan of the tile (as scan_fwd_lookback_kernel, VEC = 1)
    LaneChannels<T, 1, Off> ln;
    ln.init(g, lane, P.L, P.D, P.nch);
    ChannelConst cc[1];
    load_consts<1>(P.lam, ln.d0, cc);
    float h0v[1] = {P.h0 ? P.h0[ln.c0] : 0.0f};
    const int64_t tw = t0 + (int64_t)w * C;
    const bool full = (s + 1) * W * C <= P.L;  // workgroup-uniform
    float a[C][1], u[C][1];
    float xs[C];
#pragma unroll
    for (int j = 0; j < C; ++j) {
        const int64_t t = (full || tw + j < P.L) ? tw + j : P.L - 1;
        float v[1];
        load_vec<T, 1>((const T*)P.p0, ln.at(t), v);
        xs[j] = v[0];
    }
#pragma unroll
    for (int j = 0; j < C; ++j) {
        const bool ok = full || tw + j < P.L;
        float aj, uj;
        gate_forward<sizeof(T) == 4>(xs[j], zr[j], zi[j], cc[0], aj, uj);
        a[j][0] = ok ? aj : 1.0f;
        u[j][0] = ok ? uj : 0.0f;
    }
    {
        Seg sg{1.0f, 0.0f};
#pragma unroll
        for (int j = 0; j < C; ++j) sg = compose(Seg{a[j][0], u[j][0]}, sg);
        agg[w][lane][0] = sg;
    }
    __syncthreads();
    Seg pre = Seg{1.0f, 0.0f}, tot = Seg{1.0f, 0.0f};
#pragma unroll
    for (int q = 0; q < W; ++q) {
        const Seg e = agg[q][lane][0];
        if (q < w) pre = compose(e, pre);
        tot = compose(e, tot);
    }
    __syncthreads();
    uint64_t* const own = P.lb.states + s * P.nch + ln.c0;
    if (s == 0) {
        if (w == 0) {
            carry_sh[lane][0] = h0v[0];
            if (ln.valid) publish(own, pack_inclusive(fmaf(tot.A, h0v[0], tot.H)));
        }
    } else {
        if (w == 0 && ln.valid) publish(own, pack_aggregate(tot));
        lookback_carry<W, 1, K>(P.lb.states, P.nch, ln.c0, s, h0v, win_sh, carry_sh, w, lane,
                           P.lb.status);
        if (w == 0 && ln.valid)
            publish(own, pack_inclusive(fmaf(tot.A, carry_sh[lane][0], tot.H)));
    }
    __syncthreads();
    float hv[1] = {fmaf(pre.A, carry_sh[lane][0], pre.H)};
    if constexpr (GATED) {
        // y_t = h_t * SiLU(hz_t); h itself only if asked for.
#pragma unroll
        for (int j = 0; j < C; ++j) {
            hv[0] = fmaf(a[j][0], hv[0], u[j][0]);
            const bool ok = ln.valid && (full || tw + j < P.L);
            const int64_t t = (full || tw + j < P.L) ? tw + j : P.L - 1;
            float gz[1];
            load_vec<T, 1>((const T*)G.hz, ln.at(t), gz);
            float yv[1] = {hv[0] * fusedfwd::silu(gz[0])};
            if (ok) {
                store_vec<T, 1>((T*)G.y, ln.at(t), yv);
                if (P.h) store_vec<T, 1>((T*)P.h, ln.at(t), hv);
            }
        }
    } else {
        if (full) emit_steps<true, T, C, 1, Off>(P, ln, tw, a, u, hv);
        else emit_steps<false, T, C, 1, Off>(P, ln, tw, a, u, hv);
    }
    if (s == P.nseg - 1 && w == W - 1 && ln.valid && P.hT) P.hT[ln.c0] = hv[0];
}

// ------------------------------------------------------------------ launch plan
// Tile shapes: W waves per workgroup and E elements per lane per macro-chunk
// (C = E / VEC steps per wave), so a wave moves the same bytes per
// macro-chunk whatever VEC is.
#ifndef RECBLR_FWD_CHAIN_W
#define RECBLR_FWD_CHAIN_W 8
#endif
#ifndef RECBLR_FWD_CHAIN_E
#define RECBLR_FWD_CHAIN_E 8
#endif
#ifndef RECBLR_FWD_LB_W
#define RECBLR_FWD_LB_W 8
#endif
#ifndef RECBLR_FWD_LB_E
#define RECBLR_FWD_LB_E 16
#endif
// Channels per lane at most, per kernel (measured best on MI355X): the
// look-back kernel takes two bf16 channels per lane (4-byte accesses; a
// 2-byte access per lane streams about 10% slower) and one fp32 channel.
#ifndef RECBLR_FWD_CHAIN_MAX_VEC
#define RECBLR_FWD_CHAIN_MAX_VEC 4
#endif
#ifndef RECBLR_FWD_LB_MAX_VEC
#define RECBLR_FWD_LB_MAX_VEC 2
#endif
#ifndef RECBLR_FWD_LB_MAX_VEC_F32
#define RECBLR_FWD_LB_MAX_VEC_F32 1
#endif
constexpr int kChainW = RECBLR_FWD_CHAIN_W, kChainE = RECBLR_FWD_CHAIN_E;
constexpr int kLbW = RECBLR_FWD_LB_W, kLbE = RECBLR_FWD_LB_E;
// Look-back window per wave: K tiles, K * VEC state words per lane.
#ifndef RECBLR_FWD_LB_WORDS
#define RECBLR_FWD_LB_WORDS 1
#endif
template <int VEC>
constexpr int lb_window() { return RECBLR_FWD_LB_WORDS / VEC > 0 ? RECBLR_FWD_LB_WORDS / VEC : 1; }
template <int E, int VEC>
constexpr int steps_per_wave() { return E / VEC > 0 ? E / VEC : 1; }
// Look-back tiles keep kLbE steps per wave whatever VEC is (two channels per
// lane double the tile's channels, not its length): fewer tile rows along L
// keep the chain of inclusive states short.
template <int VEC>
constexpr int lb_steps_per_wave() { return kLbE; }
// Steps of one look-back tile.
constexpr int64_t lb_tile_steps(int) { return (int64_t)kLbW * kLbE; }
// The chain kernel is used when its workgroups alone fill the GPU.
// The chain kernel is used when its workgroups alone fill the GPU (one
// workgroup per compute unit at least); lanes then take as many channels as
// keep that many workgroups.
constexpr int64_t kChainMinGroups = 256;
// Largest channels-per-lane of a kernel for an element size (8-byte accesses
// per lane at most).
constexpr int max_vec(size_t esz, bool lookback, int64_t nch = INT64_MAX) {
    const int cap = !lookback ? RECBLR_FWD_CHAIN_MAX_VEC
                    : esz == 4 ? RECBLR_FWD_LB_MAX_VEC_F32
                               : RECBLR_FWD_LB_MAX_VEC;
    int v = (int)(8 / esz) < cap ? (int)(8 / esz) : cap;
    while (v > 1 && !lookback && nch / (kWave * v) < kChainMinGroups) v /= 2;
    return v;
}

// Channels per lane: up to max_vec, when D and the pointers allow (x-typed
// tensors aligned to VEC * esz, z-typed ones to VEC * zsz, fp32 states to
// VEC * 4).
static int pick_vec(int maxv, uintptr_t xmask, uintptr_t zmask, const float* h0, const float* hT,
                    int64_t D, size_t esz, size_t zsz) {
    const uintptr_t smask = (uintptr_t)h0 | (uintptr_t)hT;
    for (int v = maxv; v > 1; v /= 2)
        if (D % v == 0 && xmask % (v * esz) == 0 && zmask % (v * zsz) == 0 &&
            smask % (v * 4) == 0)
            return v;
    return 1;
}

struct FwdPlan {
    bool lookback;
    int vec;
    int64_t ngroups, nseg;
};

// The mode depends only on (B, L, D): the look-back kernel runs when there are
// too few channel groups for the chain kernel to fill the GPU.  The tile count
// depends on VEC (hence on pointer alignment); the workspace is sized for the
// largest VEC the mode allows (shortest tiles).
static bool forward_uses_lookback(int64_t B, int64_t L, int64_t D, size_t esz) {
    const int64_t groups_one = (B * D + kWave - 1) / kWave;
    return groups_one < kChainMinGroups && L > lb_tile_steps(max_vec(esz, true));
}

static FwdPlan plan_forward(int64_t B, int64_t L, int64_t D, size_t esz, int vec) {
    FwdPlan p;
    p.vec = vec;
    p.lookback = forward_uses_lookback(B, L, D, esz);
    p.ngroups = (B * D / vec + kWave - 1) / kWave;
    p.nseg = p.lookback ? (L + lb_tile_steps(vec) - 1) / lb_tile_steps(vec) : 1;
    return p;
}

size_t scan_forward_workspace(int64_t B, int64_t L, int64_t D, IoType io) {
    const size_t esz = io_bytes(io);
    if (!forward_uses_lookback(B, L, D, esz)) return 0;
    return lookback_ws_bytes(plan_forward(B, L, D, esz, max_vec(esz, true)).nseg, B * D);
}

// ev0 / ev1 (may be null) take the scan kernel's start and end times.
template <typename TX, typename TZ, bool RAW, typename Off, int VEC>
static hipError_t launch_vec(const FwdParams& P, const FwdPlan& plan, hipStream_t stream,
                             hipEvent_t ev0, hipEvent_t ev1) {
    if (!plan.lookback)
        return launch_measured(
            scan_fwd_chain_kernel<TX, TZ, kChainW, steps_per_wave<kChainE, VEC>(), VEC, RAW, Off>,
            dim3((unsigned)plan.ngroups), dim3(kChainW * kWave), stream, ev0, ev1, P);
    if constexpr (RAW) {
        return hipErrorInvalidValue;  // the raw scan always runs the chain kernel
    } else {
        hipError_t e = lookback_reset(P.lb, plan.nseg * P.nch, stream);
        if (e != hipSuccess) return e;
        return launch_measured(
            scan_fwd_lookback_kernel<TX, TZ, kLbW, lb_steps_per_wave<VEC>(), VEC,
                                     lb_window<VEC>(), Off>,
            dim3((unsigned)(plan.ngroups * plan.nseg)), dim3(kLbW * kWave), stream, ev0, ev1, P);
    }
}

template <typename TX, typename TZ, bool RAW>
static hipError_t launch_typed(const FwdParams& P, const FwdPlan& plan, hipStream_t stream,
                               hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr) {
    // 32-bit byte offsets whenever a whole [B, L, D] tensor spans less than 4 GiB.
    const bool small = (uint64_t)(P.nch * P.L) * sizeof(TZ) < (1ull << 32);
    // VEC = 4 only exists for 2-byte x (8-byte accesses per lane).
    if (small) {
        if constexpr (sizeof(TX) == 2)
            if (plan.vec == 4) return launch_vec<TX, TZ, RAW, uint32_t, 4>(P, plan, stream, ev0, ev1);
        if (plan.vec == 2) return launch_vec<TX, TZ, RAW, uint32_t, 2>(P, plan, stream, ev0, ev1);
        return launch_vec<TX, TZ, RAW, uint32_t, 1>(P, plan, stream, ev0, ev1);
    }
    if constexpr (sizeof(TX) == 2)
        if (plan.vec == 4) return launch_vec<TX, TZ, RAW, uint64_t, 4>(P, plan, stream, ev0, ev1);
    if (plan.vec == 2) return launch_vec<TX, TZ, RAW, uint64_t, 2>(P, plan, stream, ev0, ev1);
    return launch_vec<TX, TZ, RAW, uint64_t, 1>(P, plan, stream, ev0, ev1);
}

hipError_t launch_scan_forward(const ScanFwdArgs& a, hipStream_t stream) {
    const size_t esz = io_bytes(a.io);
    const int maxv = max_vec(esz, forward_uses_lookback(a.B, a.L, a.D, esz), a.B * a.D);
    const int vec = pick_vec(maxv, (uintptr_t)a.x | (uintptr_t)a.h,
                             (uintptr_t)a.zr | (uintptr_t)a.zi, a.h0, a.hT, a.D, esz,
                             io_bytes(a.zio));
    const FwdPlan plan = plan_forward(a.B, a.L, a.D, esz, vec);
    FwdParams P{a.x, a.zr, a.zi, a.lambda, a.h0, a.h, a.hT, a.L, a.D, a.B * a.D,
                plan.ngroups, plan.nseg, plan.lookback ? lookback_ws(a.ws) : LookbackWs{}};
    if (a.io == IoType::kF32)
        return launch_typed<float, float, false>(P, plan, stream, a.ev_begin, a.ev_end);
    if (a.zio == IoType::kF32)
        return launch_typed<bf16, float, false>(P, plan, stream, a.ev_begin, a.ev_end);
    return launch_typed<bf16, bf16, false>(P, plan, stream, a.ev_begin, a.ev_end);
}

bool fused_forward_applies(int64_t B, int64_t L, int64_t D, IoType io, const void* x,
                           const void* pack) {
    const size_t esz = io_bytes(io);
    return B > 0 && L > 0 && D > 0 && D % kWave == 0 &&
           ((uintptr_t)x | (uintptr_t)pack) % 16 == 0 &&
           (L + fastmm::BM) * D * (int64_t)esz < ((int64_t)1 << 31);
}

// Tiles of the fused forward: 64 channels x 128 steps, in tile rows along L.
static FwdPlan plan_fused(int64_t B, int64_t L, int64_t D) {
    constexpr int64_t kSteps = (int64_t)fusedz::W * fusedz::C;
    FwdPlan p;
    p.lookback = true;
    p.vec = 1;
    p.ngroups = (B * D + kWave - 1) / kWave;
    p.nseg = (L + kSteps - 1) / kSteps;
    return p;
}

size_t fused_forward_workspace(int64_t B, int64_t L, int64_t D) {
    if (B <= 0 || L <= 0 || D <= 0) return 0;
    return lookback_ws_bytes(plan_fused(B, L, D).nseg, B * D);
}

template <bool GATED>
static hipError_t launch_fused_t(const void* x, const void* pack, const void* br, const void* bi,
                                 const float* lambda, const float* h0, void* h, float* hT,
                                 int64_t B, int64_t L, int64_t D, IoType io, void* ws,
                                 const fusedfwd::GatedArgs& G, hipStream_t stream) {
    const size_t esz = io_bytes(io);
    const FwdPlan plan = plan_fused(B, L, D);
    FwdParams P{x, nullptr, nullptr, lambda, h0, h, hT, L, D, B * D, plan.ngroups, plan.nseg,
                lookback_ws(ws)};
    hipError_t e = lookback_reset(P.lb, plan.nseg * P.nch, stream);
    if (e != hipSuccess) return e;
    const dim3 grid((unsigned)(plan.ngroups * plan.nseg)), block(fusedz::NT);
    const bool small = (uint64_t)(B * L * D) * esz < (1ull << 32);
    constexpr int K = lb_window<1>();
    if (io == IoType::kF32) {
        if (small)
            hipLaunchKernelGGL((scan_fwd_fused_kernel<float, K, uint32_t, GATED>), grid, block, 0,
                               stream, P, (const __bf16*)pack, (const float*)br, (const float*)bi,
                               G);
        else
            hipLaunchKernelGGL((scan_fwd_fused_kernel<float, K, uint64_t, GATED>), grid, block, 0,
                               stream, P, (const __bf16*)pack, (const float*)br, (const float*)bi,
                               G);
    } else {
        if (small)
            hipLaunchKernelGGL((scan_fwd_fused_kernel<bf16, K, uint32_t, GATED>), grid, block, 0,
                               stream, P, (const __bf16*)pack, (const bf16*)br, (const bf16*)bi,
                               G);
        else
            hipLaunchKernelGGL((scan_fwd_fused_kernel<bf16, K, uint64_t, GATED>), grid, block, 0,
                               stream, P, (const __bf16*)pack, (const bf16*)br, (const bf16*)bi,
                               G);
    }
    return hipGetLastError();
}

hipError_t launch_fused_forward(const void* x, const void* pack, const void* br, const void* bi,
                                const float* lambda, const float* h0, void* h, float* hT,
                                int64_t B, int64_t L, int64_t D, IoType io, void* ws,
                                hipStream_t stream) {
    return launch_fused_t<false>(x, pack, br, bi, lambda, h0, h, hT, B, L, D, io, ws,
                                 fusedfwd::GatedArgs{}, stream);
}

hipError_t launch_fused_gated_forward(const void* x, const void* hz, const void* pack,
                                      const void* br, const void* bi, const float* lambda,
                                      const float* h0, void* y, void* h, float* hT, int64_t B,
                                      int64_t L, int64_t D, IoType io, void* ws,
                                      hipStream_t stream) {
    return launch_fused_t<true>(x, pack, br, bi, lambda, h0, h, hT, B, L, D, io, ws,
                                fusedfwd::GatedArgs{hz, y}, stream);
}

// Serial scan of the efficiency ablation: one wave per 64 channels walks the
// whole sequence with the state in registers (the chain kernel with a single
// wave, one channel per lane): no parallelism along the sequence.
hipError_t launch_scan_forward_serial(const ScanFwdArgs& a, hipStream_t stream) {
    const int64_t nch = a.B * a.D;
    if (nch == 0) return hipSuccess;
    const int64_t groups = (nch + kWave - 1) / kWave;
    FwdParams P{a.x, a.zr, a.zi, a.lambda, a.h0, a.h, a.hT, a.L, a.D, nch, groups, 1,
                LookbackWs{}};
    const bool small = (uint64_t)(nch * a.L) * io_bytes(a.io) < (1ull << 32);
    const dim3 grid((unsigned)groups), block(kWave);
    constexpr int C = 8;
    if (a.io == IoType::kF32) {
        if (small)
            hipLaunchKernelGGL((scan_fwd_chain_kernel<float, float, 1, C, 1, false, uint32_t>),
                               grid, block, 0, stream, P);
        else
            hipLaunchKernelGGL((scan_fwd_chain_kernel<float, float, 1, C, 1, false, uint64_t>),
                               grid, block, 0, stream, P);
    } else {
        if (small)
            hipLaunchKernelGGL((scan_fwd_chain_kernel<bf16, bf16, 1, C, 1, false, uint32_t>),
                               grid, block, 0, stream, P);
        else
            hipLaunchKernelGGL((scan_fwd_chain_kernel<bf16, bf16, 1, C, 1, false, uint64_t>),
                               grid, block, 0, stream, P);
    }
    return hipGetLastError();
}

hipError_t launch_linear_scan(const float* a, const float* u, const float* h0, float* h,
                              float* hT, int64_t B, int64_t L, int64_t D, hipStream_t stream) {
    FwdPlan plan;
    plan.lookback = false;
    plan.vec = pick_vec(max_vec(4, false, B * D), (uintptr_t)a | (uintptr_t)h, (uintptr_t)u, h0, hT,
                        D, 4, 4);
    plan.ngroups = (B * D / plan.vec + kWave - 1) / kWave;
    plan.nseg = 1;
    FwdParams P{a, u, nullptr, nullptr, h0, h, hT, L, D, B * D, plan.ngroups, 1, LookbackWs{}};
    return launch_typed<float, float, true>(P, plan, stream);
}

}  // namespace recblr
