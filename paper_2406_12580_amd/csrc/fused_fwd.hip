// Scan forward with the gate projections fused in, for D = 128 (fp32 or bf16
// I/O) and D = 256 (bf16 I/O): the gate pre-activations of section 3.2,
// z_r = W_r x_t + b_r and z_i = W_i x_t + b_i, are formed on the matrix cores
// right where the BD-LRU scan (eq:linrnn, evaluated with the operator of
// section 3.3) consumes them, so z never reaches HBM: the kernel reads x and
// writes h (or y = h * SiLU(hz), the output gate of Algorithm
// alg:gated_recurrent).
//
// Work decomposition.  A channel group is 128 consecutive channels of one
// batch row; a tile is 64 steps of a group.  A workgroup of 8 waves owns one
// group at a time; wave w owns channels 16w .. 16w + 15 of the group and
// keeps the matching rows of W_r and W_i in VGPRs for the whole launch (the
// B operand of v_mfma_f32_32x32x16_bf16: 32 columns = z_r and z_i of its 16
// channels, K = D).  Per tile:
//   * the x rows of the tile (64 steps x all D inputs) are staged into LDS by
//     16-byte direct-to-LDS loads, one tile ahead (double buffer), with the
//     16-byte chunks of each row permuted so that fragment reads do not
//     collide in LDS banks;
//   * each wave multiplies the tile's x rows (A operand, rows permuted so
//     that each lane's accumulators hold 16 consecutive steps) by its W
//     columns: two 32-step blocks, D / 16 MFMAs each (fp32 I/O: operands
//     split into bf16 hi and lo parts, three MFMAs per product);
//   * one v_permlane16_swap per pair of accumulators hands every lane z_r
//     and z_i of one channel at 8 consecutive steps: lane (rho, c) holds
//     channel c at steps 32 m + 8 rho .. + 7 of block m;
//   * the lane forms alpha and beta x (x read back from the LDS tile),
//     scans its 8 steps, and the four lanes of a channel combine their
//     segments with two cross-row swaps (permlane16 / permlane32);
//   * the tile's carry-in comes from the previous tile of the same group:
//     in registers when one workgroup walks a whole group (chain mode, at
//     least 256 groups), else by decoupled look-back over the group's tiles,
//     which workgroups bound to the group take in ticket order;
//   * h goes to an LDS tile and leaves as full 16-byte row chunks during the
//     next tile (buffer stores: steps past L are dropped by the range check).
// Each element of x is read from HBM once and each element of h written once.
#include "device_common.hpp"
#include "launch.hpp"
#include "lookback.hpp"
#include "mfma_tile.hpp"

namespace recblr {
namespace fv2 {

constexpr int TS = 64;             // steps per tile
constexpr int MB = TS / 32;        // 32-step MFMA blocks per tile
constexpr int kWindow = 8;         // look-back window, tiles
// Cache policy of the h / y stores: nontemporal (written once and read
// again only by a later backward; gated forward 291 -> 277 us at
// 256 x 2048 x 128, 308-314 -> 304 us at 16 x 16384 x 256, the plain
// layer forward unchanged).
constexpr int kOutCP = 2;
// Chain mode from this many channel groups on: one workgroup per group, and
// at least one workgroup per compute unit (two per unit for 4-wave groups).
constexpr int64_t chain_groups(int nw) { return 256 * 8 / nw; }
// Waves per workgroup (one workgroup per compute unit: the weights take 64
// VGPRs per lane at D = 256, fp32 I/O needs 64 KB more LDS for its split
// operands).  Two 4-wave workgroups per unit, whose phases could overlap,
// measured slower for bf16 at 16 x 16384 x 256 (226-251 against 217-236 us).
template <typename T>
constexpr int waves() { return 8; }
template <typename T>
constexpr int threads() { return waves<T>() * kWave; }

typedef float f16v __attribute__((ext_vector_type(16)));
typedef __bf16 b8 __attribute__((ext_vector_type(8)));
typedef __bf16 b4 __attribute__((ext_vector_type(4)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f8 __attribute__((ext_vector_type(8)));
typedef uint32_t u4v __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) void glb_void;

struct Params {
    const void* x;   // [B][L][D] I/O type
    const void* wr;  // [D][D] I/O type, [out][in]
    const void* wi;
    const void* br;  // [D] I/O type or null
    const void* bi;
    const float* lam;
    const float* h0;  // [B][D] or null
    void* h;          // [B][L][D] I/O type, or null (gated, h not kept)
    float* hT;        // [B][D] or null
    const void* hz;   // gated: [B][L][D] I/O type
    void* y;          // gated: [B][L][D] I/O type
    const float* cw4;  // conv on load: taps [4][D] (zero past K); x then holds hx
    const float* cb4;  // conv on load: bias [D]
    int64_t L, D, nch;    // nch = B * D
    int64_t ngroups, nseg;
    unsigned* counters;  // look-back mode: tile-row tickets, one per group
    uint64_t* states;    // look-back mode: [nseg][nch] state words
    unsigned* status;    // look-back mode: set when a bounded wait ran out
};

// 16-byte chunk permutations of the LDS tiles.  A bf16 row (the A operand)
// stores chunk j at position j ^ swz16(r): the 16 rows that one pass of a
// fragment read touches (rows {0..7, 16..23} or {8..15, 24..31} of a block)
// land on distinct positions.  The raw fp32 rows store chunk j at
// j ^ swz32(r), so that the four rows 8 apart that a scan read touches
// differ.
__device__ __forceinline__ int swz16(int r) { return (r & 7) | ((r >> 1) & 8); }
__device__ __forceinline__ int swz32(int r) { return ((r >> 3) & 3) << 2; }

// A-operand row of MFMA row R (0..31) in a 32-step block: rows are permuted
// so that lane half h of the 32 x 32 accumulator holds steps 16 h .. 16 h + 15
// in VGPRs 0 .. 15 (the accumulator of row 8 (v / 4) + 4 h + v % 4 is VGPR v).
__device__ __forceinline__ int sigma(int R) { return 16 * ((R >> 2) & 1) + 4 * (R >> 3) + (R & 3); }

template <typename T, int D>
struct Geo {
    static constexpr int kNW = waves<T>();          // waves per workgroup
    static constexpr int NT = kNW * kWave;          // threads
    static constexpr int CH = 16 * kNW;             // channels per group
    static constexpr bool kF32 = sizeof(T) == 4;
    static constexpr int kEsz = (int)sizeof(T);
    static constexpr int kRow = D * kEsz;            // bytes of one x row
    static constexpr int kTile = TS * kRow;          // one x tile
    static constexpr int kLoads = kTile / (NT * 16);  // 16-byte loads per thread per tile
    static constexpr int kRow16 = D * 2;             // bytes of one bf16 operand row
    static constexpr int kPlanes = kF32 ? 2 * TS * kRow16 : 0;  // hi and lo bf16 operand planes
    static constexpr int kHPitch = CH * kEsz + 16;   // LDS h tile row pitch
    static constexpr int kHTile = TS * kHPitch;
    static constexpr int kHChunks = TS * CH * kEsz / 16;  // 16-byte chunks of an h tile
    static constexpr int kSt = kHChunks / NT;        // chunks per thread
    static constexpr int kKk = D / 16;               // MFMA k-steps
    static constexpr int kSmem = 2 * kTile + kPlanes + kHTile;
    static_assert(kLoads * NT * 16 == kTile, "whole loads per tile");
    static_assert(kSt * NT == kHChunks, "whole h chunks per thread");
};

// Issues the direct-to-LDS loads of one x tile (steps t0 .. t0 + TS - 1 of
// batch row b; rows past L repeat row L - 1, which the scan masks).
template <typename T, int D>
__device__ __forceinline__ void stage_tile(const T* x, int64_t b, int64_t L, int64_t t0,
                                           char* buf, int tid, int w) {
    using G = Geo<T, D>;
    constexpr int cpr = G::kRow / 16, NT = G::NT;
#pragma unroll
    for (int q = 0; q < G::kLoads; ++q) {
        const int o = q * NT + tid;
        const int r = o / cpr, jp = o % cpr;
        const int j = jp ^ (G::kF32 ? swz32(r) : swz16(r));
        int64_t t = t0 + r;
        t = t < L ? t : L - 1;
        const char* gp = (const char*)x + ((b * L + t) * D) * G::kEsz + j * 16;
        __builtin_amdgcn_global_load_lds((const glb_void*)gp,
                                         (lds_void*)(buf + (q * NT + w * kWave) * 16), 16, 0, 0);
    }
}

// x of (local row r, input k) from the LDS tile.
template <typename T, int D>
__device__ __forceinline__ float tile_x(const char* buf, int r, int k) {
    if constexpr (sizeof(T) == 2) {
        const int off = r * (D * 2) + (((k >> 3) ^ swz16(r)) << 4) + (k & 7) * 2;
        return __uint_as_float((uint32_t)(*(const uint16_t*)(buf + off)) << 16);
    } else {
        const int off = r * (D * 4) + (((k >> 2) ^ swz32(r)) << 4) + (k & 3) * 4;
        return *(const float*)(buf + off);
    }
}

// fp32 I/O: split the raw tile into bf16 hi and lo operand planes.
template <int D, int NT>
__device__ __forceinline__ void split_tile(const char* raw, char* planes, int tid) {
    constexpr int cpr = D / 8;  // bf16 chunks per operand row
    constexpr int per = TS * cpr / NT;
#pragma unroll
    for (int q = 0; q < per; ++q) {
        const int o = q * NT + tid;
        const int r = o / cpr, jb = o % cpr;
        const f4 v0 = *(const f4*)(raw + r * (D * 4) + (((2 * jb) ^ swz32(r)) << 4));
        const f4 v1 = *(const f4*)(raw + r * (D * 4) + (((2 * jb + 1) ^ swz32(r)) << 4));
        const fastmm::u2v p0 = fastmm::split2(v0[0], v0[1]), p1 = fastmm::split2(v0[2], v0[3]);
        const fastmm::u2v p2 = fastmm::split2(v1[0], v1[1]), p3 = fastmm::split2(v1[2], v1[3]);
        const int pos = r * (D * 2) + ((jb ^ swz16(r)) << 4);
        *(u4v*)(planes + pos) = u4v{p0.x, p1.x, p2.x, p3.x};
        *(u4v*)(planes + TS * D * 2 + pos) = u4v{p0.y, p1.y, p2.y, p3.y};
    }
}

// ---- causal conv + SiLU on load (the gated layer core's input step, Algorithm
// alg:gated_recurrent): the tile's hx rows and the three rows before them are staged raw,
// x' = SiLU(b + sum_{j<4} w_j hx_{t-j}) is formed from them into the x tile
// (the layout stage_tile gives), and the products and the scan read it from
// there as from a staged x tile.
template <typename T, int D>
struct ConvGeo {
    using G = Geo<T, D>;
    static constexpr int kRows = TS + 3;             // the tile's rows and the 3 before
    static constexpr int kHx = kRows * G::kRow;       // one staged hx tile
    static constexpr int kChunks = kHx / 16;
    static constexpr int kPerWave = kChunks / G::kNW;  // 16-byte chunks per wave
    static constexpr int kLoads = (kPerWave + kWave - 1) / kWave;  // loads per wave (the last partial)
    static constexpr int kTaps = 5 * D * 4;           // [4][D] taps then [D] bias, fp32
    static constexpr int kBase = G::kTile + G::kPlanes + G::kHTile + kTaps;
    static constexpr int kLimit = 160 * 1024 - 1024;  // dynamic LDS (static slots aside)
    static constexpr int kBufs = kBase + 2 * kHx <= kLimit ? 2 : 1;  // hx tiles in LDS
    static constexpr int kSmem = kBase + kBufs * kHx;
    static constexpr int kCpr = G::kRow / 16;         // 16-byte chunks per row
    static constexpr int kRpg = TS * kCpr / G::NT;    // conv: rows per thread
    static_assert(kPerWave * G::kNW == kChunks, "hx chunks split evenly over the waves");
    static_assert(kRpg * G::NT == TS * kCpr, "conv rows split evenly over the threads");
    static_assert(kSmem <= kLimit, "LDS");
    static_assert(kConvTaps == 4, "three halo rows before the tile");
};

// Issues the direct-to-LDS loads of one hx tile: rows t0 - 3 .. t0 + TS - 1 of
// batch row b (clamped to [0, L - 1]; rows before 0 are zeroed by conv_tile),
// stored row after row.  Every wave issues ConvGeo::kLoads loads (the last
// with some lanes off), so vector-memory wait counts stay exact.
template <typename T, int D>
__device__ __forceinline__ void stage_hx(const T* hx, int64_t b, int64_t L, int64_t t0, char* buf,
                                         int lane, int w) {
    using CG = ConvGeo<T, D>;
    using G = Geo<T, D>;
#pragma unroll
    for (int q = 0; q < CG::kLoads; ++q) {
        const int c = q * kWave + lane;  // chunk within this wave's share
        if (c < CG::kPerWave) {
            const int o = w * CG::kPerWave + c;
            const int r = o / CG::kCpr, j = o % CG::kCpr;
            int64_t t = t0 - 3 + r;
            t = t < 0 ? 0 : (t < L ? t : L - 1);
            const char* gp = (const char*)hx + ((b * L + t) * D) * G::kEsz + j * 16;
            __builtin_amdgcn_global_load_lds((const glb_void*)gp,
                                             (lds_void*)(buf + (w * CG::kPerWave + q * kWave) * 16),
                                             16, 0, 0);
        }
    }
}

// x' of the tile from its staged hx rows: thread tid takes chunk tid % kCpr
// (V channels) of rows (tid / kCpr) kRpg .. + kRpg - 1, with the taps and bias
// of those channels from the LDS table.  The sum runs over j = 0 .. 3 in that
// order from the bias, as the streaming conv kernel does.
template <typename T, int D>
__device__ __forceinline__ void conv_tile(const char* hxb, const float* taps, char* xt, int64_t t0,
                                          int tid) {
    using CG = ConvGeo<T, D>;
    using G = Geo<T, D>;
    constexpr int V = 16 / (int)sizeof(T);
    constexpr int R = CG::kRpg;
    const int j = tid % CG::kCpr, r0 = (tid / CG::kCpr) * R;
    float wt[kConvTaps][V], bv[V];
#pragma unroll
    for (int v = 0; v < V; ++v) {
        bv[v] = taps[kConvTaps * D + j * V + v];
#pragma unroll
        for (int k = 0; k < kConvTaps; ++k) wt[k][v] = taps[k * D + j * V + v];
    }
    float win[R + 3][V];
#pragma unroll
    for (int i = 0; i < R + 3; ++i) {
        const u4v raw = *(const u4v*)(hxb + (r0 + i) * G::kRow + j * 16);
        const bool live = t0 - 3 + r0 + i >= 0;
#pragma unroll
        for (int v = 0; v < V; ++v) {
            float f;
            if constexpr (sizeof(T) == 2)
                f = (v & 1) ? bf16_hi(raw[v >> 1]) : bf16_lo(raw[v >> 1]);
            else
                f = __uint_as_float(raw[v]);
            win[i][v] = live ? f : 0.0f;
        }
    }
#pragma unroll
    for (int rr = 0; rr < R; ++rr) {
        const int r = r0 + rr;
        float xo[V];
#pragma unroll
        for (int v = 0; v < V; ++v) {
            float c = bv[v];
#pragma unroll
            for (int k = 0; k < kConvTaps; ++k) c = fmaf(wt[k][v], win[rr + 3 - k][v], c);
            xo[v] = c * sigmoid(c);
        }
        u4v out;
        if constexpr (sizeof(T) == 2) {
#pragma unroll
            for (int e = 0; e < 4; ++e) out[e] = bf16_pair(xo[2 * e], xo[2 * e + 1]);
            *(u4v*)(xt + r * G::kRow + ((j ^ swz16(r)) << 4)) = out;
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) out[e] = __float_as_uint(xo[e]);
            *(u4v*)(xt + r * G::kRow + ((j ^ swz32(r)) << 4)) = out;
        }
    }
}

__device__ __forceinline__ float sw_bits(uint32_t v) { return __uint_as_float(v); }

// v_permlane16_swap of two accumulators: even 16-lane rows keep a and get
// b's... see the exchange in the kernel.
__device__ __forceinline__ void swap16(float& a, float& b) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a), __float_as_uint(b), false,
                                                    false);
    a = __uint_as_float(r[0]);
    b = __uint_as_float(r[1]);
}
// The value of the lane in the neighbouring 16-lane row (rows 0 <-> 1, 2 <-> 3).
__device__ __forceinline__ float row_partner(float v, bool odd) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                    false);
    return __uint_as_float(odd ? r[0] : r[1]);
}
// The value of the lane 32 away (lower half <-> upper half).
__device__ __forceinline__ float half_partner(float v, bool upper) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                    false);
    return __uint_as_float(upper ? r[0] : r[1]);
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes,
                                             0x00020000);
}

__device__ __forceinline__ float silu(float c) { return c * sigmoid(c); }

// gate_forward on pre-activations that still lack their biases: the exponent
// of each sigmoid is formed as fma(z, -log2 e, nb) with nb = -b log2 e, so
// adding the bias costs no instruction (z + b is never rounded on its own).
template <bool kSeries = true>
__device__ __forceinline__ void gate_forward_biased(float x, float zr, float zi, float nbr,
                                                    float nbi, const ChannelConst& cc,
                                                    float& alpha, float& u) {
    float r = fast_rcp(1.0f + fast_exp2(fmaf(zr, -kLog2e, nbr)));
    float i = fast_rcp(1.0f + fast_exp2(fmaf(zi, -kLog2e, nbi)));
    alpha = fast_exp2(r * cc.neg_s_l2);
    float m = kSeries ? one_minus_exp_neg(r * cc.two_s, alpha) : fmaf(-alpha, alpha, 1.0f);
    u = fast_sqrt(m) * i * x;
}

// Workgroup barrier for LDS hand-offs that leaves vector-memory operations in
// flight: __syncthreads() carries a release fence, which waits for every
// outstanding load and store of the wave (the direct-to-LDS prefetch of the
// next tile among them).  Here the wave's own LDS writes are waited for
// (lgkmcnt(0)), and direct-to-LDS loads are waited for explicitly (vmcnt)
// before the barrier that publishes their data; the empty asm statements keep
// the compiler from moving memory accesses across the barrier.
__device__ __forceinline__ void lds_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt and expcnt not waited for
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// s_waitcnt immediate that waits until at most n vector-memory operations of
// the wave are outstanding (lgkmcnt and expcnt not waited for).
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | 0x0F70; }

// The 16-byte chunks of one h tile that thread tid writes: output (and, gated,
// hz input) byte offsets within batch row b's [L][D] block.
template <typename T, int D>
__device__ __forceinline__ uint32_t chunk_offset(int64_t t0, int64_t cg, int q, int tid) {
    using G = Geo<T, D>;
    constexpr int cpr = G::CH * G::kEsz / 16;
    const int o = q * G::NT + tid;
    const int r = o / cpr, c = o % cpr;
    return (uint32_t)(((t0 + r) * D + cg * G::CH) * G::kEsz + c * 16);
}

// Element-wise y = h * SiLU(hz) on one 16-byte chunk.
template <typename T>
__device__ __forceinline__ u4v gate_chunk(u4v hv, u4v zv) {
    u4v out;
    if constexpr (sizeof(T) == 4) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
            out[e] = __float_as_uint(__uint_as_float(hv[e]) * silu(__uint_as_float(zv[e])));
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
            out[e] = bf16_pair(bf16_lo(hv[e]) * silu(bf16_lo(zv[e])),
                               bf16_hi(hv[e]) * silu(bf16_hi(zv[e])));
    }
    return out;
}

// CONV (gated only): x holds hx and x' = SiLU(conv(hx)) is formed on load.
template <typename T, int D, bool GATED, bool LOOKBACK, bool CONV = false>
__global__ __launch_bounds__(threads<T>(), 2) void fused_fwd_kernel(Params P) {
    using G = Geo<T, D>;
    using CG = ConvGeo<T, D>;
    constexpr int NT = G::NT, CH = G::CH;
    extern __shared__ __attribute__((aligned(16))) char smem[];
    __shared__ int64_t slot_sh[2];
    // LDS: two x tiles (double buffer), the bf16 operand planes (fp32 I/O),
    // the h tile; with CONV one x' tile, the planes, the h tile, the conv
    // taps and one or two staged hx tiles.
    char* const xbuf0 = smem;
    char* const xbuf1 = CONV ? smem : smem + G::kTile;
    char* const planes = smem + (CONV ? 1 : 2) * G::kTile;
    char* const hst = planes + G::kPlanes;
    float* const taps = (float*)(hst + G::kHTile);
    char* const hxbuf0 = hst + G::kHTile + CG::kTaps;
    char* const hxbuf1 = CG::kBufs == 2 ? hxbuf0 + CG::kHx : hxbuf0;

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int w = wave_id();
    const int rho = lane >> 4;         // 16-lane row
    const bool odd = rho & 1, upper = rho >= 2;

    // ---- group of this workgroup
    int64_t g;
    if constexpr (LOOKBACK) {
        g = blockIdx.x % P.ngroups;
    } else {
        g = blockIdx.x;
    }
    const int64_t gpr = P.D / CH;  // groups per batch row
    const int64_t b = g / gpr, cg = g - b * gpr;
    const int cw = (int)cg * CH + 16 * w;  // first input-channel index of this wave
    const int cl = lane & 15;              // channel of this lane within the wave
    const int64_t chan = b * P.D + cw + cl;  // flat channel of this lane

    // ---- tile rows: chain mode walks 0 .. nseg-1; look-back mode takes tickets
    int64_t s_cur, s_next;
    if constexpr (LOOKBACK) {
        if (tid == 0) {
            slot_sh[0] = (int64_t)atomicAdd(P.counters + g, 1u);
            slot_sh[1] = (int64_t)atomicAdd(P.counters + g, 1u);
        }
        __syncthreads();
        s_cur = slot_sh[0];
        s_next = slot_sh[1];
    } else {
        s_cur = 0;
        s_next = 1;
    }
    if (s_cur >= P.nseg) return;

    // ---- W columns of this wave in VGPRs (B operand): lane l holds column
    // l % 32 (z_r of channel cw + l % 16 for l % 32 < 16, else z_i) at
    // k = 16 kk + 8 (l / 32) .. + 7.
    const int col = lane & 31;
    const T* wsrc = (const T*)(col < 16 ? P.wr : P.wi) + (int64_t)(cw + (col & 15)) * D;
    b8 wf[G::kKk];
    b8 wl[G::kF32 ? G::kKk : 1];
#pragma unroll
    for (int kk = 0; kk < G::kKk; ++kk) {
        const int k0 = 16 * kk + 8 * (lane >> 5);
        if constexpr (G::kF32) {
            const f4 a = *(const f4*)(wsrc + k0);
            const f4 c = *(const f4*)(wsrc + k0 + 4);
            const f8 v = {a[0], a[1], a[2], a[3], c[0], c[1], c[2], c[3]};
            wf[kk] = __builtin_convertvector(v, b8);
            wl[G::kF32 ? kk : 0] = __builtin_convertvector(v - __builtin_convertvector(wf[kk], f8), b8);
        } else {
            wf[kk] = *(const b8*)(wsrc + k0);
        }
    }
    // Biases of this lane's channel cw + cl (after the swap below a lane holds
    // z_r and z_i of one channel), folded into the sigmoids' exponents.
    const float nbr = P.br ? -load((const T*)P.br + cw + cl) * kLog2e : 0.0f;
    const float nbi = P.bi ? -load((const T*)P.bi + cw + cl) * kLog2e : 0.0f;
    const ChannelConst cc = channel_const(P.lam[cw + cl]);
    // LDS byte offsets of this lane's x in a tile (local rows 8 rho + i; block
    // m adds 32 m rows): the chunk permutation of row 32 m + 8 rho + i is
    // i | 8 [rho >= 2] for bf16 rows and 4 rho for fp32 rows.
    int xoff[sizeof(T) == 2 ? 8 : 1];
    {
        const int k = cw + cl;
        if constexpr (sizeof(T) == 2) {
#pragma unroll
            for (int i = 0; i < 8; ++i)
                xoff[i] = (8 * rho + i) * G::kRow + (((k >> 3) ^ (i | (rho >= 2 ? 8 : 0))) << 4) +
                          (k & 7) * 2;
        } else {
            xoff[0] = 8 * rho * G::kRow + (((k >> 2) ^ (4 * rho)) << 4) + (k & 3) * 4;
        }
    }
    float carry = P.h0 ? P.h0[chan] : 0.0f;  // chain mode: state before the current tile

    const T* xg = (const T*)P.x;
    const uint32_t row_bytes = (uint32_t)(P.L * P.D * G::kEsz);
    const __amdgpu_buffer_rsrc_t hr = rsrc((const char*)P.h + b * P.L * P.D * G::kEsz,
                                           P.h ? row_bytes : 0u);
    const __amdgpu_buffer_rsrc_t yr =
        rsrc(GATED ? (const char*)P.y + b * P.L * P.D * G::kEsz : nullptr, GATED ? row_bytes : 0u);
    const __amdgpu_buffer_rsrc_t zr_ =
        rsrc(GATED ? (const char*)P.hz + b * P.L * P.D * G::kEsz : nullptr,
             GATED ? row_bytes : 0u);
    u4v hz_load[GATED ? G::kSt : 1], hz_store[GATED ? G::kSt : 1];

    if constexpr (CONV) {
        // the taps table, visible after the loop's first barrier
        for (int i = tid; i < 5 * D; i += NT)
            taps[i] = i < kConvTaps * D ? P.cw4[i] : P.cb4[i - kConvTaps * D];
        stage_hx<T, D>(xg, b, P.L, s_cur * TS, hxbuf0, lane, w);
    } else {
        stage_tile<T, D>(xg, b, P.L, s_cur * TS, xbuf0, tid, w);
    }

    int64_t s_prev = -1;  // tile whose h waits in the LDS h tile
    constexpr int kHz = GATED ? G::kSt : 0;  // hz loads per thread per tile
    // Loads of the next tile issued at the top of an iteration (x, or hx with
    // two hx buffers; a single hx buffer is refilled after the conv instead).
    constexpr bool kEarly = !CONV || CG::kBufs == 2;
    constexpr int kNextLoads = CONV ? CG::kLoads : G::kLoads;
    for (int64_t it = 0;; ++it) {
        char* const cur = (it & 1) ? xbuf1 : xbuf0;
        char* const nxt = (it & 1) ? xbuf0 : xbuf1;
        char* const hxcur = (it & 1) ? hxbuf1 : hxbuf0;
        char* const hxnxt = (it & 1) ? hxbuf0 : hxbuf1;
        lds_barrier();  // all waves are done with the previous tile: nxt is free, hst is full
        const bool has_next = s_next < P.nseg;
        unsigned ticket = 0;
        if constexpr (LOOKBACK) {
            if (tid == 0) ticket = atomicAdd(P.counters + g, 1u);  // the tile after next
        }
        if constexpr (GATED) {
            // hz of the previous tile (loaded one iteration ago) for its y.
#pragma unroll
            for (int q = 0; q < G::kSt; ++q) hz_store[q] = hz_load[q];
        }
        if (kEarly && has_next) {
            if constexpr (CONV)
                stage_hx<T, D>(xg, b, P.L, s_next * TS, hxnxt, lane, w);
            else
                stage_tile<T, D>(xg, b, P.L, s_next * TS, nxt, tid, w);
        }
        if constexpr (GATED) {
            // hz of the current tile, used when its h leaves (next iteration).
#pragma unroll
            for (int q = 0; q < G::kSt; ++q)
                hz_load[q] = __builtin_amdgcn_raw_buffer_load_b128(
                    zr_, chunk_offset<T, D>(s_cur * TS, cg, q, tid), 0, 0);
        }
        // Everything but the loads just issued has landed: the current tile's
        // x (or hx) rows, issued one iteration ago, among it.
        if (kEarly && has_next)
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(kNextLoads + kHz));
        else
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(kHz));
        // ---- the previous tile's h (and y) leave in 16-byte row chunks
        if (s_prev >= 0) {
            constexpr int cpr = CH * G::kEsz / 16;
#pragma unroll
            for (int q = 0; q < G::kSt; ++q) {
                const int o = q * NT + tid;
                const u4v hv = *(const u4v*)(hst + (o / cpr) * G::kHPitch + (o % cpr) * 16);
                const uint32_t off = chunk_offset<T, D>(s_prev * TS, cg, q, tid);
                if constexpr (GATED) {
                    __builtin_amdgcn_raw_buffer_store_b128(gate_chunk<T>(hv, hz_store[q]), yr, off,
                                                           0, kOutCP);
                }
                __builtin_amdgcn_raw_buffer_store_b128(hv, hr, off, 0, kOutCP);
            }
        }
        if constexpr (LOOKBACK) {
            if (tid == 0) slot_sh[it & 1] = (int64_t)ticket;
        }
        lds_barrier();  // the current tile is in LDS for every wave; the h tile is free
        const int64_t s = s_cur;
        const int64_t t0 = s * TS;
        if constexpr (CONV) {
            conv_tile<T, D>(hxcur, taps, cur, t0, tid);
            lds_barrier();  // x' is in LDS for every wave; hxcur is free
            if (!kEarly && has_next) stage_hx<T, D>(xg, b, P.L, s_next * TS, hxbuf0, lane, w);
        }
        const char* abuf = cur;
        if constexpr (G::kF32) {
            split_tile<D, NT>(cur, planes, tid);
            lds_barrier();
            abuf = planes;
        }

        // ---- z = x W^T for 64 steps x this wave's 32 columns (b comes with the gates)
        f16v acc[MB];
#pragma unroll
        for (int m = 0; m < MB; ++m)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[m][v] = 0.0f;
        {
            const int R = lane & 31;
#pragma unroll
            for (int kk = 0; kk < G::kKk; ++kk) {
                const int j = 2 * kk + (lane >> 5);
#pragma unroll
                for (int m = 0; m < MB; ++m) {
                    const int r = 32 * m + sigma(R);
                    const int pos = r * G::kRow16 + ((j ^ swz16(r)) << 4);
                    const b8 a = *(const b8*)(abuf + pos);
                    if constexpr (G::kF32) {
                        const b8 alo = *(const b8*)(abuf + TS * G::kRow16 + pos);
                        acc[m] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, wl[G::kF32 ? kk : 0],
                                                                        acc[m], 0, 0, 0);
                        acc[m] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(alo, wf[kk], acc[m], 0,
                                                                        0, 0);
                    }
                    acc[m] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, wf[kk], acc[m], 0, 0, 0);
                }
            }
        }
        // ---- hand every lane z_r and z_i of channel cl at steps 32 m + 8 rho + i
#pragma unroll
        for (int m = 0; m < MB; ++m)
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                float zr = acc[m][i], zi = acc[m][i + 8];
                swap16(zr, zi);
                acc[m][i] = zr;
                acc[m][i + 8] = zi;
            }

        // ---- gates (alpha into acc[m][i], beta' into acc[m][i + 8]) and segments.
        // Only the last tile can hold rows past L (they become the identity);
        // the full tiles take a path without the per-element masks.
        Seg run[MB];
        const int lim = P.L - t0 < TS ? (int)(P.L - t0) : TS;  // valid rows of the tile
        auto gates = [&](auto full_tag) {
            constexpr bool kFull = decltype(full_tag)::value;
#pragma unroll
            for (int m = 0; m < MB; ++m) {
                Seg sg{1.0f, 0.0f};
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    float xv;
                    if constexpr (sizeof(T) == 2)
                        xv = __uint_as_float((uint32_t)(*(const uint16_t*)(cur + xoff[i] +
                                                                           32 * m * G::kRow))
                                             << 16);
                    else
                        xv = *(const float*)(cur + xoff[0] + (32 * m + i) * G::kRow);
                    float a, u;
                    gate_forward_biased<sizeof(T) == 4>(xv, acc[m][i], acc[m][i + 8], nbr, nbi,
                                                        cc, a, u);
                    if constexpr (!kFull) {
                        const bool ok = 32 * m + 8 * rho + i < lim;
                        a = ok ? a : 1.0f;
                        u = ok ? u : 0.0f;
                    }
                    acc[m][i] = a;
                    acc[m][i + 8] = u;
                    sg = Seg{a * sg.A, fmaf(a, sg.H, u)};
                }
                run[m] = sg;
            }
        };
        if (lim == TS)
            gates(std::true_type{});
        else
            gates(std::false_type{});
        // ---- the four runs of a block: exclusive prefix and block total
        Seg excl[MB], tot[MB];
#pragma unroll
        for (int m = 0; m < MB; ++m) {
            const Seg p{row_partner(run[m].A, odd), row_partner(run[m].H, odd)};
            const Seg pair = odd ? compose(run[m], p) : compose(p, run[m]);
            const Seg e1 = odd ? p : Seg{1.0f, 0.0f};
            const Seg o{half_partner(pair.A, upper), half_partner(pair.H, upper)};
            tot[m] = upper ? compose(pair, o) : compose(o, pair);
            excl[m] = upper ? compose(e1, o) : e1;
        }
        Seg tile{1.0f, 0.0f};
#pragma unroll
        for (int m = 0; m < MB; ++m) tile = compose(tot[m], tile);

        // ---- carry into the tile
        float cin;
        if constexpr (LOOKBACK) {
            uint64_t* const own = P.states + s * P.nch + chan;
            const float h0v = P.h0 ? P.h0[chan] : 0.0f;
            if (s == 0) {
                cin = h0v;
            } else {
                if (rho == 0) publish(own, pack_aggregate(tile));
                uint64_t wd[kWindow];
#pragma unroll
                for (int j = 0; j < kWindow; ++j) {
                    const int64_t p = s - 1 - j;
                    wd[j] = p >= 0 ? peek(P.states + p * P.nch + chan) : pack_inclusive(h0v);
                }
#pragma unroll
                for (int j = 0; j < kWindow; ++j) {
                    const int64_t p = s - 1 - j;
                    if (p >= 0) wd[j] = wait_ready(P.states + p * P.nch + chan, wd[j], P.status);
                }
                const int64_t oldest = s - kWindow;
                cin = fold_window<kWindow>(wd, P.states + (oldest >= 0 ? oldest : 0) * P.nch + chan,
                                           P.status);
            }
            if (rho == 0) publish(own, pack_inclusive(fmaf(tile.A, cin, tile.H)));
        } else {
            cin = carry;
            carry = fmaf(tile.A, cin, tile.H);
        }
        if (s == P.nseg - 1 && rho == 0 && P.hT) P.hT[chan] = fmaf(tile.A, cin, tile.H);

        // ---- h of the lane's steps into the LDS h tile
        float cm = cin;
#pragma unroll
        for (int m = 0; m < MB; ++m) {
            float hv = fmaf(excl[m].A, cm, excl[m].H);
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                hv = fmaf(acc[m][i], hv, acc[m][i + 8]);
                char* dst = hst + (32 * m + 8 * rho + i) * G::kHPitch + (16 * w + cl) * G::kEsz;
                if constexpr (sizeof(T) == 4)
                    *(float*)dst = hv;
                else
                    *(uint16_t*)dst = from_f32<bf16>(hv).bits;
            }
            cm = fmaf(tot[m].A, cm, tot[m].H);
        }

        s_prev = s;
        s_cur = s_next;
        if constexpr (LOOKBACK) {
            s_next = slot_sh[it & 1];
        } else {
            s_next = s_cur + 1;
        }
        if (s_cur >= P.nseg) break;
    }
    lds_barrier();  // the last tile's h is in LDS
    {
        constexpr int cpr = CH * G::kEsz / 16;
#pragma unroll
        for (int q = 0; q < G::kSt; ++q) {
            const int o = q * NT + tid;
            const u4v hv = *(const u4v*)(hst + (o / cpr) * G::kHPitch + (o % cpr) * 16);
            const uint32_t off = chunk_offset<T, D>(s_prev * TS, cg, q, tid);
            if constexpr (GATED) {
                __builtin_amdgcn_raw_buffer_store_b128(gate_chunk<T>(hv, hz_load[q]), yr, off, 0,
                                                       kOutCP);
            }
            __builtin_amdgcn_raw_buffer_store_b128(hv, hr, off, 0, kOutCP);
        }
    }
}

// Look-back workspace: a 256-byte header (status word at byte 4, as in the
// other look-back kernels), ngroups tile counters (256-byte aligned), then
// [nseg][nch] state words.
struct Plan {
    bool lookback;
    int64_t ngroups, nseg;
};

inline int waves_of(IoType io) { return io == IoType::kF32 ? waves<float>() : waves<bf16>(); }

inline Plan plan(int64_t B, int64_t L, int64_t D, int nw) {
    Plan p;
    p.ngroups = B * D / (16 * nw);
    p.nseg = (L + TS - 1) / TS;
    p.lookback = p.ngroups < chain_groups(nw) && p.nseg > 1;
    return p;
}

inline size_t counters_bytes(int64_t ngroups) {
    return ((size_t)ngroups * sizeof(unsigned) + 255) / 256 * 256;
}

__global__ void reset_kernel(unsigned* __restrict__ counters, int64_t ngroups,
                             uint64_t* __restrict__ states, int64_t n, unsigned* status) {
    const int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    if (i0 == 0) *status = 0u;
    for (int64_t i = i0; i < ngroups; i += stride) counters[i] = 0u;
    for (int64_t i = i0; i < n; i += stride) states[i] = ~0ull;
}

template <typename T, int D, bool GATED, bool LOOKBACK, bool CONV>
hipError_t launch(const Params& P, int grid, hipStream_t stream) {
    auto kern = fused_fwd_kernel<T, D, GATED, LOOKBACK, CONV>;
    constexpr int smem = CONV ? ConvGeo<T, D>::kSmem : Geo<T, D>::kSmem, nt = Geo<T, D>::NT;
    static const hipError_t attr =
        hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, smem);
    if (attr != hipSuccess) return attr;
    hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(nt), smem, stream, P);
    return hipGetLastError();
}

template <typename T, int D, bool GATED, bool CONV = false>
hipError_t launch_mode(const Params& P, const Plan& pl, hipStream_t stream) {
    if (!pl.lookback) return launch<T, D, GATED, false, CONV>(P, (int)pl.ngroups, stream);
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus < 1)
        cus = 256;
    // Workgroups bound to each group; they take the group's tiles in ticket order.
    const int64_t slots = (int64_t)cus * (8 / Geo<T, D>::kNW);
    int64_t per = (slots + pl.ngroups - 1) / pl.ngroups;
    if (per > pl.nseg) per = pl.nseg;
    return launch<T, D, GATED, true, CONV>(P, (int)(pl.ngroups * per), stream);
}

}  // namespace fv2

bool fused2_forward_applies(int64_t B, int64_t L, int64_t D, IoType io, const void* x,
                            const void* wr, const void* wi) {
    const size_t esz = io_bytes(io);
    const bool shape = io == IoType::kF32 ? D == 128 : (D == 128 || D == 256);
    return B > 0 && L > 0 && shape && ((uintptr_t)x | (uintptr_t)wr | (uintptr_t)wi) % 16 == 0 &&
           (L + fv2::TS) * D * (int64_t)esz < ((int64_t)1 << 31) &&
           B * D < ((int64_t)1 << 40);
}

size_t fused2_forward_workspace(int64_t B, int64_t L, int64_t D, IoType io) {
    if (B <= 0 || L <= 0 || D <= 0 || D % 128 != 0) return 0;
    const fv2::Plan p = fv2::plan(B, L, D, fv2::waves_of(io));
    if (!p.lookback) return 0;
    return 256 + fv2::counters_bytes(p.ngroups) + (size_t)(p.nseg * B * D) * sizeof(uint64_t);
}

hipError_t launch_fused2_forward(const void* x, const void* wr, const void* br, const void* wi,
                                 const void* bi, const float* lambda, const float* h0, void* h,
                                 float* hT, const void* hz, void* y, int64_t B, int64_t L,
                                 int64_t D, IoType io, void* ws, hipStream_t stream,
                                 const float* w4, const float* b4) {
    const fv2::Plan pl = fv2::plan(B, L, D, fv2::waves_of(io));
    fv2::Params P{x,  wr,        wi,  br,  bi,  lambda, h0, h, hT, hz, y, w4, b4, L, D, B * D,
                  pl.ngroups, pl.nseg, nullptr, nullptr, nullptr};
    if (pl.lookback) {
        P.status = (unsigned*)((char*)ws + kStatusOffset);
        P.counters = (unsigned*)((char*)ws + 256);
        P.states = (uint64_t*)((char*)ws + 256 + fv2::counters_bytes(pl.ngroups));
        const int64_t n = pl.nseg * B * D;
        int64_t blocks = (n + 255) / 256;
        blocks = blocks > 1024 ? 1024 : (blocks < 1 ? 1 : blocks);
        hipLaunchKernelGGL(fv2::reset_kernel, dim3((unsigned)blocks), dim3(256), 0, stream,
                           P.counters, pl.ngroups, P.states, n, P.status);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const bool gated = y != nullptr;
    if (w4 && (!gated || !b4)) return hipErrorInvalidValue;  // conv on load: gated layer only
    if (w4) {
        if (io == IoType::kF32) return fv2::launch_mode<float, 128, true, true>(P, pl, stream);
        if (D == 128) return fv2::launch_mode<bf16, 128, true, true>(P, pl, stream);
        return fv2::launch_mode<bf16, 256, true, true>(P, pl, stream);
    }
    if (io == IoType::kF32)
        return gated ? fv2::launch_mode<float, 128, true>(P, pl, stream)
                     : fv2::launch_mode<float, 128, false>(P, pl, stream);
    if (D == 128)
        return gated ? fv2::launch_mode<bf16, 128, true>(P, pl, stream)
                     : fv2::launch_mode<bf16, 128, false>(P, pl, stream);
    return gated ? fv2::launch_mode<bf16, 256, true>(P, pl, stream)
                 : fv2::launch_mode<bf16, 256, false>(P, pl, stream);
}

}  // namespace recblr
