// Cross-workgroup carry propagation for the chunked BD-LRU scans
// (decoupled look-back over the scan operator of RecBLR, arXiv 2406.12580,
// section 3.3).
//
// When a sequence is split into tiles handled by different workgroups, every
// tile publishes, per channel, one 64-bit state word:
//   high 32 bits  0xFFFFFFFF             not ready yet
//                 bit 31 set             aggregate: A = bits & 0x7FFFFFFF, low word = H
//                 bit 31 clear           inclusive: low word = the state after the tile
//   low 32 bits   H or the inclusive state (fp32 bits)
// A is a product of decay factors in [0, 1], so its sign bit is free; a NaN A
// is published as A = 1 with H = NaN so that the NaN still propagates.  The
// word is written and read with relaxed agent-scope 64-bit atomics (single
// global_store/load_dwordx2 with the coherence bit, no fence): status and
// payload travel together, so no release/acquire ordering is needed.
//
// Tiles are handed out in ticket order (an atomic counter), so the tile a
// workgroup waits on was taken by a workgroup that is already running and
// publishes its aggregate without waiting on anyone: the wait always ends.
// Spins are still bounded; an exhausted bound yields NaN instead of a hang
// and sets a status word in the workspace header, so that the caller can tell
// it from a NaN that came with the inputs.
#pragma once

#include "device_common.hpp"

namespace recblr {

constexpr uint32_t kNotReady = 0xFFFFFFFFu;
constexpr uint32_t kAggBit = 0x80000000u;
constexpr int kSpinLimit = 1 << 20;

__device__ __forceinline__ uint64_t pack_aggregate(Seg s) {
    float A = s.A, H = s.H;
    if (A != A) {
        A = 1.0f;
        H = __uint_as_float(0x7FC00000u);
    }
    return ((uint64_t)(__float_as_uint(A) | kAggBit) << 32) | __float_as_uint(H);
}

__device__ __forceinline__ uint64_t pack_inclusive(float h) {
    return (uint64_t)__float_as_uint(h);
}

__device__ __forceinline__ uint32_t word_status(uint64_t w) { return (uint32_t)(w >> 32); }
__device__ __forceinline__ bool word_ready(uint64_t w) { return word_status(w) != kNotReady; }
__device__ __forceinline__ bool word_inclusive(uint64_t w) {
    return (word_status(w) & kAggBit) == 0u;
}
__device__ __forceinline__ Seg word_aggregate(uint64_t w) {
    return Seg{__uint_as_float(word_status(w) & ~kAggBit), __uint_as_float((uint32_t)w)};
}
__device__ __forceinline__ float word_value(uint64_t w) { return __uint_as_float((uint32_t)w); }

__device__ __forceinline__ void publish(uint64_t* p, uint64_t w) {
    __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint64_t peek(const uint64_t* p) {
    return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
}

// Records in the workspace status word that a bounded wait ran out.
__device__ __forceinline__ void flag_exhausted(unsigned* status) {
    if (status) __hip_atomic_fetch_or(status, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Wait until the word at p is ready (bounded); returns it, or a NaN inclusive
// word (and sets *status) if the bound runs out.
__device__ __forceinline__ uint64_t wait_ready(const uint64_t* p, uint64_t w, unsigned* status) {
    int spins = 0;
    while (!word_ready(w)) {
        if (++spins > kSpinLimit) {
            flag_exhausted(status);
            return pack_inclusive(__uint_as_float(0x7FC00000u));
        }
        __builtin_amdgcn_s_sleep(1);
        w = peek(p);
    }
    return w;
}

// Carry from the state words of tiles r-1 .. r-N of one channel (wd[i] is
// tile r-1-i, all ready): starting from the nearest inclusive state, the
// aggregates after it are applied oldest first.  If none of the N is
// inclusive, waits (bounded) for tile r-N's inclusive state at `oldest`.
// Unrolled with selects: no dynamic indexing, no branches but the wait.
template <int N>
__device__ __forceinline__ float fold_window(uint64_t (&wd)[N], const uint64_t* oldest,
                                             unsigned* status) {
    int nearest = N;
#pragma unroll
    for (int i = N - 1; i >= 0; --i)
        if (word_inclusive(wd[i])) nearest = i;
    if (nearest == N) {
        // None of the N is inclusive yet: wait for the oldest to be.  (Waiting
        // for tile r-1 instead would chain the tiles one after another
        // whenever more than N tile rows are in flight.)
        uint64_t w = wd[N - 1];
        int spins = 0;
        while (!word_inclusive(w)) {
            if (++spins > kSpinLimit) {
                flag_exhausted(status);
                w = pack_inclusive(__uint_as_float(0x7FC00000u));
                break;
            }
            __builtin_amdgcn_s_sleep(1);
            w = peek(oldest);
        }
        wd[N - 1] = w;
        nearest = N - 1;
    }
    float v = 0.0f;
#pragma unroll
    for (int i = N - 1; i >= 0; --i) {
        const Seg e = word_aggregate(wd[i]);
        const float f = fmaf(e.A, v, e.H);
        v = i == nearest ? word_value(wd[i]) : (i < nearest ? f : v);
    }
    return v;
}

// Carry into tile r (tile index in processing order) from the state words of
// tiles < r, bitwise reproducibly.
//
// Every tile q publishes incl(q) = fma(A_q, carry_in(q), H_q) with (A_q, H_q)
// its own aggregate.  The carry into r is formed the same way: starting from
// the nearest published inclusive state incl(p), the aggregates of tiles
// p+1 .. r-1 are applied one at a time, oldest first, with the same fma.  By
// induction the result is bitwise incl(r-1) whichever p is found, so the
// output does not depend on the timing of the other workgroups.
//
// All W waves call this.  Wave q reads the window of tiles
// r-1-q*K .. r-q*K-K (waiting until each word is ready) into LDS; wave 0
// then finds the nearest inclusive state and applies the aggregates after it.
// If the W*K tiles read hold no inclusive state, wave 0 waits for the oldest
// of them, tile r-W*K, to publish its inclusive state, and folds the others
// onto it; so a tile never waits on the tile right before it, and the chain
// of waits advances W*K tiles at a time.  Tiles before tile 0 stand for `init`.
// Leaves the carry of every lane in carry_sh.
template <int W, int VEC, int K>
__device__ __forceinline__ void lookback_carry(const uint64_t* __restrict__ states, int64_t nch,
                                               int64_t c0, int64_t r, const float (&init)[VEC],
                                               uint64_t (&win_sh)[W * K][kWave][VEC],
                                               float (&carry_sh)[kWave][VEC], int w, int lane,
                                               unsigned* status) {
    // Issue all K*VEC loads of the window first, then wait on any not ready.
    uint64_t wv[K][VEC];
#pragma unroll
    for (int j = 0; j < K; ++j) {
        const int64_t p = r - 1 - (int64_t)w * K - j;
#pragma unroll
        for (int k = 0; k < VEC; ++k)
            wv[j][k] = p >= 0 ? peek(states + p * nch + c0 + k) : pack_inclusive(init[k]);
    }
#pragma unroll
    for (int j = 0; j < K; ++j) {
        const int64_t p = r - 1 - (int64_t)w * K - j;
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
            if (p >= 0) wv[j][k] = wait_ready(states + p * nch + c0 + k, wv[j][k], status);
            win_sh[w * K + j][lane][k] = wv[j][k];
        }
    }
    __syncthreads();
    if (w == 0) {
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
            uint64_t wd[W * K];
#pragma unroll
            for (int i = 0; i < W * K; ++i) wd[i] = win_sh[i][lane][k];
            carry_sh[lane][k] = fold_window<W * K>(wd, states + (r - W * K) * nch + c0 + k, status);
        }
    }
}

// Fills the state words with "not ready" and zeroes the ticket counter and
// the status word (internal linkage: every translation unit launches its own
// copy).
static __global__ void lookback_init_kernel(uint64_t* __restrict__ states, int64_t n,
                                            unsigned* __restrict__ ticket) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < 2) ticket[i] = 0u;  // ticket, status
    for (int64_t k = i; k < n; k += (int64_t)gridDim.x * blockDim.x) states[k] = ~0ull;
}

// Workspace of a look-back launch: a 256-byte header holding the ticket
// counter (byte 0) and the status word (byte 4: nonzero once a bounded wait
// ran out), then one state word per (tile, channel).
constexpr size_t kStatusOffset = 4;
struct LookbackWs {
    unsigned* ticket;
    unsigned* status;
    uint64_t* states;
};

inline size_t lookback_ws_bytes(int64_t nseg, int64_t nch) {
    return 256 + (size_t)(nseg * nch) * sizeof(uint64_t);
}

inline LookbackWs lookback_ws(void* ws) {
    return LookbackWs{(unsigned*)ws, (unsigned*)((char*)ws + kStatusOffset),
                      (uint64_t*)((char*)ws + 256)};
}

inline hipError_t lookback_reset(const LookbackWs& w, int64_t n, hipStream_t stream) {
    int64_t blocks = (n + 255) / 256;
    if (blocks > 1024) blocks = 1024;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(lookback_init_kernel, dim3((unsigned)blocks), dim3(256), 0, stream,
                       w.states, n, w.ticket);
    return hipGetLastError();
}

}  // namespace recblr
