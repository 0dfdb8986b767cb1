// Gate pre-activations of one scan tile on the matrix cores (RecBLR,
// arXiv 2406.12580, section 3.2: z_r = W_r x_t + b_r, z_i = W_i x_t + b_i).
//
// A tile is 64 channels (channel group cg of batch row b) x 128 steps.  Its
// pre-activations for both gates are one 128 x 128 product
//   [z_r | z_i](steps t0 .. t0+127, the group's 64 channels each)
//     = x[b, t0 .. t0+127, 0 .. D-1] . [W_r; W_i](group)^T + [b_r; b_i]
// with K = D, on bf16 MFMA tiles with fp32 accumulation (fp32 operands take
// the 3-term bf16 split of the fastmm engine).  Wave w of 8 computes the
// 16 x 128 strip of steps t0+16w .. t0+16w+15 and turns it into the
// lane-per-channel layout of the scan kernels through a wave-private LDS
// strip: lane l receives channel cg*64 + l's 16 values of each gate.
// Used by the fused forward and backward scans, so that z never reaches HBM.
#pragma once

#include "device_common.hpp"
#include "mfma_tile.hpp"

namespace recblr {
namespace fusedz {

constexpr int W = 8, C = 16;   // waves; steps per wave (tile = 128 steps)
constexpr int NT = W * kWave;  // threads
constexpr int ZP = 20;         // z strip pitch (floats) per column: 16 steps + 4

// Wave w's 16 x 128 strip of the staged slices: rows 16 w .. 16 w + 15 of A,
// all 128 rows of B, k-steps of 32 (lane l supplies row l % 16 and
// k = 8 (l / 16) .. +7 of each fragment).
template <int PA, int PB>
__device__ __forceinline__ void strip_mma(__bf16 (*la)[fastmm::BM][fastmm::KP],
                                          __bf16 (*lb)[fastmm::BN][fastmm::KP], fastmm::f4 (&acc)[8],
                                          int w, int lane) {
    using namespace fastmm;
    const int fr = lane & 15, fk = 8 * (lane >> 4);
#pragma unroll
    for (int ks = 0; ks < BK; ks += 32) {
        const int ra = 16 * w + fr;
        b8 fa[PA];
#pragma unroll
        for (int p = 0; p < PA; ++p) fa[p] = *(const b8*)&la[p][ra][lds_col(ra, ks + fk)];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int rb = 16 * j + fr;
            b8 fb[PB];
#pragma unroll
            for (int p = 0; p < PB; ++p) fb[p] = *(const b8*)&lb[p][rb][lds_col(rb, ks + fk)];
            if constexpr (PB == 2)
                acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[0], fb[1], acc[j], 0, 0, 0);
            if constexpr (PA == 2)
                acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[1], fb[0], acc[j], 0, 0, 0);
            acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[0], fb[0], acc[j], 0, 0, 0);
        }
    }
}

// Operand kinds and LDS size of the tile product for x of type T and weights
// of type TW (bf16 weights are one exact plane even against fp32 x: the
// split's hi * lo term would only add zeros).
template <typename T, typename TW = T>
struct Tile {
    static constexpr bool kF32 = sizeof(T) == 4;
    using OpA = fastmm::Operand<kF32 ? fastmm::kF32 : fastmm::kBf16, true>;
    using OpB = fastmm::Operand<sizeof(TW) == 4 ? fastmm::kPack2 : fastmm::kPack1, true>;
    static constexpr int PA = OpA::kPlanes, PB = OpB::kPlanes;
    static constexpr size_t kStage =
        (size_t)(PA * fastmm::BM + PB * fastmm::BN) * fastmm::KP * 2;
    static constexpr size_t kZ = (size_t)W * 64 * ZP * sizeof(float);
    static constexpr size_t kSmem = kStage > kZ ? kStage : kZ;
};

// z_r, z_i of the tile for this lane's channel at this wave's 16 steps.
// x: [B][L][D] (row b is read), pack: [W_r; W_i] of type TW ordered by
// channel group of 64 (launch_pack_groups), biases (TW) may be null;
// D % 64 == 0.  Steps past L read x as zero.  smem: Tile<T, TW>::kSmem
// bytes, free on entry; all NT threads call this (it holds workgroup
// barriers).
template <typename T, typename TW = T>
__device__ __forceinline__ void tile_z(const T* x, const __bf16* pack, const TW* br,
                                       const TW* bi, int64_t L, int64_t D, int64_t b,
                                       int64_t cg, int64_t t0, char* smem, int tid, int w,
                                       int lane, float (&zr)[C], float (&zi)[C]) {
    using namespace fastmm;
    using TT = Tile<T, TW>;
    using OpA = typename TT::OpA;
    using OpB = typename TT::OpB;
    constexpr int PA = TT::PA, PB = TT::PB;
    f4 acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    {
        __bf16 (*la)[BM][KP] = (__bf16 (*)[BM][KP])smem;
        __bf16 (*lb)[BN][KP] = (__bf16 (*)[BN][KP])(smem + (size_t)PA * BM * KP * 2);
        const uint32_t plane = (uint32_t)(2 * D * D * 2);
        const OpA a{resource(x + b * L * D, (uint32_t)(L * D * sizeof(T))),
                    (uint32_t)(D * sizeof(T)), 0, 0, 0};
        const OpB wb{resource(pack + cg * 128 * D, (PB - 1) * plane + (uint32_t)(128 * D * 2)),
                     (uint32_t)(D * 2), 0, 0, plane};
        const Stager<OpB, NT> sb(wb, 0, tid);
        typename OpB::raw_t rb[quads<NT>()];
        const int64_t nsl = (D + BK - 1) / BK;
        sb.fetch(wb, 0, D, tid, rb);
        constexpr int Q = quads<NT>();
        const Stager<OpA, NT> sa(a, t0, tid);
        typename OpA::raw_t ra[Q];
        sa.fetch(a, 0, D, tid, ra);
        for (int64_t sl = 0; sl < nsl; ++sl) {
            store_slice<OpA, NT>(la, tid, ra);
            store_slice<OpB, NT>(lb, tid, rb);
            __syncthreads();
            if (sl + 1 < nsl) {
                sa.fetch(a, (sl + 1) * BK, D, tid, ra);
                sb.fetch(wb, (sl + 1) * BK, D, tid, rb);
            }
            __builtin_amdgcn_sched_barrier(0);
            strip_mma<PA, PB>(la, lb, acc, w, lane);
            __syncthreads();
        }
    }
    // Bias, then the strip to the lane-per-channel layout, one gate at a time
    // through a wave-private LDS strip of 64 columns: column c (16 consecutive
    // steps) becomes lane c's z_r, then its z_i.  A wave's LDS operations
    // execute in order, so the second gate may reuse the strip.
    float* zs = (float*)smem + w * 64 * ZP;
    const ElemReader<TW> rbr(br, D), rbi(bi, D);
    const int64_t d = cg * kWave + (lane & 15);
#pragma unroll
    for (int gate = 0; gate < 2; ++gate) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int col = 16 * j + (lane & 15);
            const float bias = gate == 0 ? rbr(d + 16 * j) : rbi(d + 16 * j);
            *(f4*)&zs[col * ZP + 4 * (lane >> 4)] = acc[4 * gate + j] + f4{bias, bias, bias, bias};
        }
        float* dst = gate == 0 ? zr : zi;
#pragma unroll
        for (int q = 0; q < C / 4; ++q) {
            const f4 v = *(const f4*)&zs[lane * ZP + 4 * q];
#pragma unroll
            for (int e = 0; e < 4; ++e) dst[4 * q + e] = v[e];
        }
    }
}

}  // namespace fusedz
}  // namespace recblr
