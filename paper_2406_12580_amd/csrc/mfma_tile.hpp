// Staging engine of the bf16 matrix-core tiles (gfx950): operands read
// through buffer resources as quads of 4 consecutive elements, fp32 values
// split into bf16 hi and lo planes, and 128 x BK slices kept in LDS with a
// swizzled layout for conflict-free fragment reads.  Used by the gate
// projections (gemm.hip) and by the scan forward with the projections fused
// in (scan_fwd.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device_common.hpp"

namespace recblr {
namespace fastmm {
constexpr int BM = 128, BN = 128, BK = 64;
// Quads (4 consecutive elements) per thread and operand in one 128 x BK
// slice staged by NT threads.
template <int NT>
constexpr int quads() {
    return BM * BK / 4 / NT;
}
constexpr int NQ = quads<256>();
// LDS tiles hold BK bf16 per row (128 bytes); the 16-byte chunk j of row r is
// stored at chunk j ^ f(r) with f(r) = (r ^ (r >> 2)) mod 8, so that the
// fragment reads (8 consecutive rows, one chunk) and the transposed stores
// (rows 4m + c for consecutive m, one chunk) each touch 8 distinct chunk
// positions.
constexpr int KP = BK;
constexpr uint32_t kOOB = 0x80000000u;  // at or past every resource size: loads return 0

typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f8 __attribute__((ext_vector_type(8)));
typedef __bf16 b4 __attribute__((ext_vector_type(4)));
typedef __bf16 b8 __attribute__((ext_vector_type(8)));
typedef uint32_t u2v __attribute__((ext_vector_type(2)));
typedef uint32_t u4v __attribute__((ext_vector_type(4)));

// Column (bf16 elements) at which element k of LDS row `row` is stored.
__device__ __forceinline__ int lds_col(int row, int k) {
    const int f = (row ^ (row >> 2)) & 7;
    return (((k >> 3) ^ f) << 3) | (k & 7);
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t resource(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes,
                                             0x00020000);
}

__device__ __forceinline__ f4 widen(f4 v) { return v; }
__device__ __forceinline__ f4 widen(u2v v) {
    return f4{__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u),
              __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xffff0000u)};
}
// Element c of four packed bf16 as 16 bits.
__device__ __forceinline__ uint32_t bits16(u2v v, int c) {
    const uint32_t w = c < 2 ? v.x : v.y;
    return (c & 1) ? w >> 16 : w & 0xffffu;
}

// {hi, lo}: hi = bf16(a) and lo = bf16(a - hi), and the same for b, as
// packed bf16 pairs (round to nearest even).  hi's halves are widened back
// by a shift and a mask; written as a conversion of the vector, the
// compiler converts every value a second time on its own to widen it (4
// instructions per value instead of 3).
__device__ __forceinline__ u2v split2(float a, float b) {
    const uint32_t hi = bf16_pair(a, b);
    return u2v{hi, bf16_pair(a - __uint_as_float(hi << 16), b - __uint_as_float(hi & 0xffff0000u))};
}

// Kinds of operand data.
enum Kind {
    kF32,    // fp32 values, split into hi and lo planes on the way to LDS
    kBf16,   // bf16 values, one plane
    kPack1,  // packed weights: one bf16 plane
    kPack2,  // packed weights: bf16 hi and lo planes
};

template <int KIND>
struct RawOf {
    using type = u2v;
};
template <>
struct RawOf<kF32> {
    using type = f4;
};
template <>
struct RawOf<kPack2> {
    struct type {
        u2v p[2];
    };
};

// Operand with element (mn, k): mn is the output row (A) or column (B), k the
// contracted index.  KFAST: memory rows are mn and k runs along them;
// otherwise memory rows are k.  Byte offset of memory element (row, col):
// row * pitch + col_off(col), where PAIR operands hold columns [0, half) at
// byte 0 and [half, 2 half) at byte hoff (the two gates' fp32 scratch).
template <int KIND, bool KFAST, bool PAIR = false>
struct Operand {
    static constexpr int kKind = KIND;
    static constexpr bool kKFast = KFAST;
    static constexpr int kPlanes = (KIND == kF32 || KIND == kPack2) ? 2 : 1;
    static constexpr uint32_t kEsz = KIND == kF32 ? 4 : 2;
    using raw_t = typename RawOf<KIND>::type;
    __amdgpu_buffer_rsrc_t rsrc;
    uint32_t pitch;  // bytes per memory row
    uint32_t half;   // PAIR: columns per half
    uint32_t hoff;   // PAIR: byte offset of the second half
    uint32_t plane;  // kPack2: bytes per plane
    __device__ uint32_t col_off(int64_t c) const {
        if constexpr (PAIR)
            return c < half ? (uint32_t)c * 4u : hoff + (uint32_t)(c - half) * 4u;
        else
            return (uint32_t)c * kEsz;
    }
    __device__ uint32_t row_off(int64_t r) const {
        const uint64_t o = (uint64_t)r * pitch;
        return o < kOOB ? (uint32_t)o : kOOB;
    }
    __device__ raw_t load(uint32_t off) const {
        if constexpr (KIND == kF32) {
            const u4v v = __builtin_amdgcn_raw_buffer_load_b128(rsrc, off, 0, 0);
            return f4{__uint_as_float(v.x), __uint_as_float(v.y), __uint_as_float(v.z),
                      __uint_as_float(v.w)};
        } else if constexpr (KIND == kPack2) {
            raw_t r;
            r.p[0] = __builtin_amdgcn_raw_buffer_load_b64(rsrc, off, 0, 0);
            r.p[1] = __builtin_amdgcn_raw_buffer_load_b64(rsrc, off + plane, 0, 0);
            return r;
        } else {
            return __builtin_amdgcn_raw_buffer_load_b64(rsrc, off, 0, 0);
        }
    }
};

// Per-thread staging of one operand's 128 x BK slices by NT threads, Q =
// quads<NT>() quads per thread:
//   KFAST: quad j covers (mn = tid / 16 + (NT / 16) j, k = 4 (tid % 16) .. +3).
//   else : (NT = 256) quad j covers (mn = 4 (tid % 32) .. +3, k = NQ (tid / 32) + j).
// The per-tile part of the byte offsets is fixed at construction; quad j
// adds j times a uniform stride (NT / 16 memory rows, or one memory row).
// The launch bounds keep every in-tile row offset below 2^31.
template <class Op, int NT = 256>
struct Stager {
    static constexpr int Q = quads<NT>();
    static_assert(Op::kKFast || NT == 256, "transposed staging is laid out for 256 threads");
    uint32_t fixed;
    __device__ Stager(const Op& op, int64_t mn0, int tid) {
        if constexpr (Op::kKFast)
            fixed = op.row_off(mn0 + (tid >> 4));
        else
            fixed = op.col_off(mn0 + 4 * (tid & 31));
    }
    // Loads the slice starting at k0 (zeros for k >= k_end).
    __device__ void fetch(const Op& op, int64_t k0, int64_t k_end, int tid,
                          typename Op::raw_t (&r)[Q]) const {
        if constexpr (Op::kKFast) {
            const int64_t k = k0 + 4 * (tid & 15);
            const uint32_t base = fixed + (k < k_end ? op.col_off(k) : kOOB);
            const uint32_t step = (NT / 16) * op.pitch;
#pragma unroll
            for (int j = 0; j < Q; ++j) r[j] = op.load(base + j * step);
        } else {
            const int64_t k = k0 + Q * (tid >> 5);
            const uint32_t base = op.row_off(k) + fixed;
            if (k0 + BK <= k_end) {
#pragma unroll
                for (int j = 0; j < Q; ++j) r[j] = op.load(base + j * op.pitch);
            } else {
#pragma unroll
                for (int j = 0; j < Q; ++j)
                    r[j] = op.load(k + j < k_end ? base + j * op.pitch : kOOB);
            }
        }
    }
};

template <int N>
struct PackT;
template <>
struct PackT<8> {
    using bits = uint4;
    using fv = f8;
    using bv = b8;
};

// Writes a slice staged by NT threads to the operand's LDS planes.
template <class Op, int NT = 256>
__device__ __forceinline__ void store_slice(__bf16 (*lds)[BM][KP], int tid,
                                            const typename Op::raw_t (&r)[quads<NT>()]) {
    constexpr int KIND = Op::kKind;
    if constexpr (Op::kKFast) {
#pragma unroll
        for (int j = 0; j < quads<NT>(); ++j) {
            const int row = (tid >> 4) + (NT / 16) * j, col = lds_col(row, 4 * (tid & 15));
            if constexpr (KIND == kF32) {
                const f4 v = r[j];
                const u2v p = split2(v[0], v[1]), q = split2(v[2], v[3]);
                *(u2v*)&lds[0][row][col] = u2v{p.x, q.x};
                *(u2v*)&lds[1][row][col] = u2v{p.y, q.y};
            } else if constexpr (KIND == kPack2) {
                *(u2v*)&lds[0][row][col] = r[j].p[0];
                *(u2v*)&lds[1][row][col] = r[j].p[1];
            } else {
                *(u2v*)&lds[0][row][col] = r[j];  // bf16 bits as they are
            }
        }
    } else {
        static_assert(KIND == kF32 || KIND == kBf16, "transposed staging of packed weights");
        // Transpose in registers: column c of the thread's quads becomes NQ
        // consecutive k of LDS row 4 mq + c.
        using PK = PackT<NQ>;
        const int mq = tid & 31, kc = NQ * (tid >> 5);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int row = 4 * mq + c, col = lds_col(row, kc);
            if constexpr (KIND == kBf16) {
                uint32_t w[NQ / 2];
#pragma unroll
                for (int j = 0; j < NQ / 2; ++j)
                    w[j] = bits16(r[2 * j], c) | (bits16(r[2 * j + 1], c) << 16);
                *(typename PK::bits*)&lds[0][row][col] = *(const typename PK::bits*)w;
            } else {
                uint32_t hi[NQ / 2], lo[NQ / 2];
#pragma unroll
                for (int j = 0; j < NQ / 2; ++j) {
                    const u2v p = split2(r[2 * j][c], r[2 * j + 1][c]);
                    hi[j] = p.x;
                    lo[j] = p.y;
                }
                *(typename PK::bits*)&lds[0][row][col] = *(const typename PK::bits*)hi;
                *(typename PK::bits*)&lds[1][row][col] = *(const typename PK::bits*)lo;
            }
        }
    }
}

// Column sums over k of a non-KFAST operand's staged slice (used for db):
// thread (mq, kg) adds its NQ k values of each of its four columns.
template <class Raw>
__device__ __forceinline__ void add_colsum(f4& cs, const Raw (&r)[NQ]) {
    f4 t = widen(r[0]);
#pragma unroll
    for (int j = 1; j < NQ; ++j) t += widen(r[j]);
    cs += t;
}

// Reads element i of a length-n array through a buffer resource (a null
// array reads as zeros, as does any i past its end): no branch, so the
// compiler need not wait for it early.
template <typename T>
struct ElemReader {
    __amdgpu_buffer_rsrc_t rsrc;
    __device__ ElemReader(const T* p, int64_t n)
        : rsrc(resource(p, p ? (uint32_t)(n * sizeof(T)) : 0u)) {}
    __device__ float operator()(int64_t i) const {
        const uint32_t off = i >= 0 && i < (int64_t)(kOOB / sizeof(T)) ? (uint32_t)(i * sizeof(T))
                                                                       : kOOB;
        if constexpr (sizeof(T) == 4) {
            return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rsrc, off, 0, 0));
        } else {
            const uint32_t b = __builtin_amdgcn_raw_buffer_load_b16(rsrc, off, 0, 0);
            return __uint_as_float(b << 16);
        }
    }
};

}  // namespace fastmm
}  // namespace recblr
