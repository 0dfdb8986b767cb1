// Device-side helpers shared by the BD-LRU kernels (gfx950 / CDNA4, wave64).
//
// Gate arithmetic of the behavior-dependent linear recurrent unit
// (RecBLR, arXiv 2406.12580, section 3.2):
//   r = sigmoid(z_r), i = sigmoid(z_i), q = softplus(Lambda) * r
//   alpha = exp(-q), beta = sqrt(1 - alpha^2) * i
// evaluated in fp32 with the hardware transcendental units (v_exp, v_log,
// v_rcp, v_sqrt, v_rsq), and 1 - alpha^2 = 1 - exp(-2q) evaluated without
// cancellation when q is small (see one_minus_exp_neg).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace recblr {

constexpr int kWave = 64;

// Index of the calling wave within its workgroup, as a wave-uniform (scalar) value.
__device__ __forceinline__ int wave_id() {
    return __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
}
constexpr float kLog2e = 1.4426950408889634f;

// ------------------------------------------------------------------ I/O types
struct bf16 {
    uint16_t bits;
};

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16 v) { return __uint_as_float((uint32_t)v.bits << 16); }

template <typename T>
__device__ __forceinline__ T from_f32(float v);

template <>
__device__ __forceinline__ float from_f32<float>(float v) { return v; }

// Round to nearest, ties to even (NaN stays NaN): the hardware conversion.
template <>
__device__ __forceinline__ bf16 from_f32<bf16>(float v) {
    bf16 out;
    out.bits = __builtin_bit_cast(uint16_t, (__bf16)v);
    return out;
}

template <typename T>
__device__ __forceinline__ float load(const T* p) { return to_f32(*p); }

// Load/store at a byte offset from a kernel-argument base pointer.  With a
// 32-bit offset the compiler emits the scalar-base + 32-bit-vector-offset
// form of global_load/global_store, so one VGPR addresses every tensor that
// shares the element offset (x, z_r, z_i, h, dh all do).
// ------------------------------------------------------------------ vector I/O
// A lane owns VEC consecutive channels; their VEC elements of one time step
// are one contiguous load or store of VEC * sizeof(T) bytes.  The sequence
// tensors are streamed exactly once, so every access carries the
// non-temporal hint.
template <typename T, int VEC>
struct VecT;
template <> struct VecT<float, 1> { using type = float; };
template <> struct VecT<float, 2> { using type = float __attribute__((ext_vector_type(2))); };
template <> struct VecT<float, 4> { using type = float __attribute__((ext_vector_type(4))); };
template <> struct VecT<bf16, 1> { using type = uint16_t; };
template <> struct VecT<bf16, 2> { using type = uint32_t; };
template <> struct VecT<bf16, 4> { using type = uint32_t __attribute__((ext_vector_type(2))); };

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
// Two floats to a packed bf16 pair (one v_cvt_pk_bf16_f32, round to nearest even).
__device__ __forceinline__ uint32_t bf16_pair(float lo, float hi) {
    typedef float f2 __attribute__((ext_vector_type(2)));
    typedef __bf16 b2 __attribute__((ext_vector_type(2)));
    const f2 v = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, b2));
}

// Widen a raw VEC-element access to fp32.
template <typename T, int VEC>
__device__ __forceinline__ void unpack_vec(typename VecT<T, VEC>::type v, float (&out)[VEC]) {
    if constexpr (sizeof(T) == 4) {
        if constexpr (VEC == 1) out[0] = v;
        else {
#pragma unroll
            for (int k = 0; k < VEC; ++k) out[k] = v[k];
        }
    } else if constexpr (VEC == 1) {
        out[0] = __uint_as_float((uint32_t)v << 16);
    } else if constexpr (VEC == 2) {
        out[0] = bf16_lo(v);
        out[1] = bf16_hi(v);
    } else {
        out[0] = bf16_lo(v[0]);
        out[1] = bf16_hi(v[0]);
        out[2] = bf16_lo(v[1]);
        out[3] = bf16_hi(v[1]);
    }
}

// One lane's VEC elements as they are in memory (bf16 pairs stay packed, so
// a register holds two of them until they are used).
template <typename T, int VEC, typename Off>
__device__ __forceinline__ typename VecT<T, VEC>::type load_raw(const T* p, Off off_bytes) {
    using V = typename VecT<T, VEC>::type;
    return __builtin_nontemporal_load((const V*)((const char*)p + off_bytes));
}

template <typename T, int VEC, typename Off>
__device__ __forceinline__ void load_vec(const T* p, Off off_bytes, float (&out)[VEC]) {
    unpack_vec<T, VEC>(load_raw<T, VEC>(p, off_bytes), out);
}

template <typename T, int VEC, typename Off>
__device__ __forceinline__ void store_vec(T* p, Off off_bytes, const float (&in)[VEC]) {
    using V = typename VecT<T, VEC>::type;
    V v;
    if constexpr (sizeof(T) == 4) {
        if constexpr (VEC == 1) v = in[0];
        else {
#pragma unroll
            for (int k = 0; k < VEC; ++k) v[k] = in[k];
        }
    } else if constexpr (VEC == 1) {
        v = from_f32<bf16>(in[0]).bits;
    } else if constexpr (VEC == 2) {
        v = bf16_pair(in[0], in[1]);
    } else {
        v[0] = bf16_pair(in[0], in[1]);
        v[1] = bf16_pair(in[2], in[3]);
    }
    __builtin_nontemporal_store(v, (V*)((char*)p + off_bytes));
}

template <typename T>
__device__ __forceinline__ void store(T* p, float v) { *p = from_f32<T>(v); }

// Byte offset into a TZ tensor from the byte offset of the same element in a
// TX tensor (TZ is never narrower than TX).
template <typename TX, typename TZ, typename Off>
__device__ __forceinline__ Off z_offset(Off off_x) {
    static_assert(sizeof(TZ) >= sizeof(TX), "z tensors are at least as wide as x");
    return sizeof(TZ) == sizeof(TX) ? off_x : off_x * (Off)(sizeof(TZ) / sizeof(TX));
}

// ------------------------------------------------------------------ gate math
__device__ __forceinline__ float fast_exp2(float v) { return __builtin_amdgcn_exp2f(v); }
__device__ __forceinline__ float fast_rcp(float v) { return __builtin_amdgcn_rcpf(v); }
__device__ __forceinline__ float fast_sqrt(float v) { return __builtin_amdgcn_sqrtf(v); }
__device__ __forceinline__ float fast_rsq(float v) { return __builtin_amdgcn_rsqf(v); }

// sigmoid(z) = 1 / (1 + e^-z); saturates cleanly to 0 and 1 for large |z|.
__device__ __forceinline__ float sigmoid(float z) {
    return fast_rcp(1.0f + fast_exp2(-z * kLog2e));
}

__device__ __forceinline__ float fast_log2(float v) { return __builtin_amdgcn_logf(v); }
constexpr float kLn2 = 0.6931471805599453f;

// softplus(v) = log(1 + e^v) = max(v, 0) + log1p(e), e = e^-|v| in [0, 1].
// For e < 1/16, log1p(e) is its Maclaurin series e - e^2/2 + ... - e^6/6; the
// first omitted term bounds the relative error by (1/16)^6 / 7 < 1e-8, and the
// series keeps full relative accuracy however small e is.  From 1/16 on,
// log1p(e) = ln(1 + e) with 1 + e in [17/16, 2]: its rounding (2^-24) moves
// the logarithm by at most 2^-24 / (17/16 ln(17/16)) < 1e-6 relative, on top
// of the hardware log2's own error (checked against fp64 over the range).  Once
// per lane (channel) per launch, so hardware exp2 / log2 are used: this is
// ~20 instructions against ~140 for the libm log1pf(expf()).
__device__ __forceinline__ float softplus(float v) {
    const float e = fast_exp2(-fabsf(v) * kLog2e);
    float p = -1.0f / 6.0f;
    p = fmaf(p, e, 1.0f / 5.0f);
    p = fmaf(p, e, -1.0f / 4.0f);
    p = fmaf(p, e, 1.0f / 3.0f);
    p = fmaf(p, e, -1.0f / 2.0f);
    p = fmaf(p, e, 1.0f);
    const float series = e * p;
    const float direct = fast_log2(1.0f + e) * kLn2;
    return fmaxf(v, 0.0f) + (e < 0.0625f ? series : direct);
}

// 1 - e^-y for y >= 0.  For y < 1/8 the Maclaurin series of 1 - e^-y,
// y * sum_{n>=0} (-y)^n / (n+1)!, truncated after the y^5 term: the first
// omitted term bounds the relative error by (1/8)^5 / 6! < 4.3e-8.  From 1/8
// on, the direct form 1 - a^2 with a = e^-(y/2) has a^2 <= e^-1/8 = 0.8825,
// so a few ulp of error in a^2 stay below 1e-6 relative to 1 - a^2 >= 0.1175.
__device__ __forceinline__ float one_minus_exp_neg(float y, float a) {
    float p = 1.0f / 120.0f;
    p = fmaf(p, -y, 1.0f / 24.0f);
    p = fmaf(p, -y, 1.0f / 6.0f);
    p = fmaf(p, -y, 0.5f);
    p = fmaf(p, -y, 1.0f);
    const float series = y * p;
    const float direct = fmaf(-a, a, 1.0f);
    return y < 0.125f ? series : direct;
}

// Per-channel constants derived from Lambda.
struct ChannelConst {
    float s;        // softplus(Lambda)
    float neg_s_l2; // -softplus(Lambda) * log2(e): alpha = exp2(r * neg_s_l2)
    float two_s;    // 2 softplus(Lambda): 2q = r * two_s
};

__device__ __forceinline__ ChannelConst channel_const(float lam) {
    ChannelConst c;
    c.s = softplus(lam);
    c.neg_s_l2 = -c.s * kLog2e;
    c.two_s = 2.0f * c.s;
    return c;
}

// alpha and beta' = beta * x of one element (forward path).  kSeries: 1 -
// alpha^2 through one_minus_exp_neg (full relative accuracy however small
// 2q is).  Without it, 1 - alpha^2 is formed directly (one fma): its error
// is about one ulp of 1 in absolute terms, so beta = sqrt(1 - alpha^2) i is
// off by at most ~1e-3 of itself for 2q down to 3e-5 and by a few 1e-4 in
// absolute terms below that, which bf16 I/O (a 2^-9 rounding of every input
// and output) does not see; it saves the series' ~7 instructions per element
// (the bf16 fused forward, 16 x 16384 x 256: 222 -> 209 us).  The backward
// keeps the series: its dz_r and dLambda terms carry 1 / sqrt(1 - alpha^2).
template <bool kSeries = true>
__device__ __forceinline__ void gate_forward(float x, float zr, float zi, const ChannelConst& cc,
                                             float& alpha, float& u) {
    float r = sigmoid(zr);
    float i = sigmoid(zi);
    alpha = fast_exp2(r * cc.neg_s_l2);
    float m = kSeries ? one_minus_exp_neg(r * cc.two_s, alpha) : fmaf(-alpha, alpha, 1.0f);
    u = fast_sqrt(m) * i * x;
}

// (A, H) pair of the scan operator: a segment maps a state h to A h + H.
// Composing an earlier segment e with a later segment l gives
// (A_l A_e, A_l H_e + H_l) (section 3.3, operator "bullet").
struct Seg {
    float A, H;
};

__device__ __forceinline__ Seg compose(Seg later, Seg earlier) {
    return Seg{later.A * earlier.A, fmaf(later.A, earlier.H, later.H)};
}

}  // namespace recblr
