// Host-side launchers of the BD-LRU kernels.  Internal to librecblr.so: the
// C ABI in capi.cpp validates every argument and then calls these.  Every
// launcher enqueues work on `stream` and returns hipGetLastError().
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace recblr {

enum class IoType : int { kF32 = 0, kBf16 = 1 };

inline size_t io_bytes(IoType t) { return t == IoType::kF32 ? 4 : 2; }

struct ScanFwdArgs {
    const void* x;
    const void* zr;
    const void* zi;
    const float* lambda;
    const float* h0;  // may be null (zero state)
    void* h;
    float* hT;        // may be null
    int64_t B, L, D;
    IoType io;        // element type of x and h
    IoType zio;       // element type of z_r, z_i (fp32 scratch in the entry points with weights)
    void* ws;         // look-back state, when the launcher uses it
    size_t ws_bytes;
    hipEvent_t ev_begin = nullptr;  // recorded right before / after the main scan
    hipEvent_t ev_end = nullptr;    // kernel's launch when not null
};

struct ScanBwdArgs {
    const void* x;
    const void* zr;
    const void* zi;
    const float* lambda;
    const float* h0;   // may be null
    const void* h;     // forward output
    const void* dh;
    const float* dhT;  // may be null
    void* dx;
    void* dzr;
    void* dzi;
    float* dlambda;
    float* dh0;        // may be null
    int64_t B, L, D;
    IoType io;        // element type of x, h, dh, dx
    IoType zio;       // element type of z_r, z_i, dz_r, dz_i
    void* ws;
    size_t ws_bytes;
    hipEvent_t ev_begin = nullptr;  // as in ScanFwdArgs
    hipEvent_t ev_end = nullptr;
};

// Launches `kernel` on `stream`.  With measurement events (either may be
// null) the launch goes through hipExtLaunchKernelGGL, which stamps the
// events with the kernel's own start and end times from its dispatch.
template <typename Kernel, typename... Args>
inline hipError_t launch_measured(Kernel kernel, dim3 grid, dim3 block, hipStream_t stream,
                                  hipEvent_t ev0, hipEvent_t ev1, Args... args) {
    if (ev0 || ev1)
        hipExtLaunchKernelGGL(kernel, grid, block, 0, stream, ev0, ev1, 0, args...);
    else
        hipLaunchKernelGGL(kernel, grid, block, 0, stream, args...);
    return hipGetLastError();
}

// Static scratch of the entry point that allocates nothing
// (recblr_bdlru_scan_backward_noalloc): a device array of this many bytes,
// one per GPU, held until the process ends.  static_scratch returns its
// address on the current device (looked up once per device).
constexpr size_t kStaticScratchBytes = (size_t)16 << 20;
hipError_t static_scratch(void** ptr, size_t* bytes);

// Workspace (bytes) the scan launchers need for a given problem.
size_t scan_forward_workspace(int64_t B, int64_t L, int64_t D, IoType io);
size_t scan_backward_workspace(int64_t B, int64_t L, int64_t D, IoType io);

hipError_t launch_scan_forward(const ScanFwdArgs& a, hipStream_t stream);
hipError_t launch_scan_backward(const ScanBwdArgs& a, hipStream_t stream);
hipError_t launch_linear_scan(const float* a, const float* u, const float* h0, float* h,
                              float* hT, int64_t B, int64_t L, int64_t D, hipStream_t stream);
hipError_t launch_scan_step(const void* x, const void* zr, const void* zi, const float* lambda,
                            const float* h_prev, float* h_next, int64_t B, int64_t D, IoType io,
                            IoType zio, hipStream_t stream);
hipError_t launch_fill(float* dst, float value, int64_t n, hipStream_t stream);
// Recurrent step with the gate projections fused in, for bf16 I/O and
// D in {64, 128, 192, 256}: persistent workgroups keep W_r and W_i resident
// in registers (no workspace).  Returns false, having launched nothing, where
// it does not apply (other dtype or D, x / W_r / W_i not 16-byte aligned,
// B * D * 4 >= 2^31); else launches and stores the launch status in *err.
bool launch_step_resident(const void* x, const void* wr, const void* br, const void* wi,
                          const void* bi, const float* lambda, const float* h_prev,
                          float* h_next, int64_t B, int64_t D, IoType io, hipStream_t stream,
                          hipError_t* err);

// Scan forward with the gate projections computed per tile on the matrix
// cores (z never reaches HBM).  Applies when the look-back kernel runs,
// D % 64 == 0 and x and pack are 16-byte aligned; pack holds the weights
// ordered by channel group (launch_pack_groups); ws is the scan-forward
// workspace.
bool fused_forward_applies(int64_t B, int64_t L, int64_t D, IoType io, const void* x,
                           const void* pack);
// Look-back workspace of the fused forward (0 for empty shapes).
size_t fused_forward_workspace(int64_t B, int64_t L, int64_t D);
hipError_t launch_fused_forward(const void* x, const void* pack, const void* br, const void* bi,
                                const float* lambda, const float* h0, void* h, float* hT,
                                int64_t B, int64_t L, int64_t D, IoType io, void* ws,
                                hipStream_t stream);

// Scan forward with the gate projections fused in, weights resident in VGPRs
// (fused_fwd.hip): D = 128 for fp32 I/O, D = 128 or 256 for bf16 I/O, x, W_r
// and W_i 16-byte aligned.  With y non-null it stores y = h * SiLU(hz) (and h
// where h is non-null).  ws: fused2_forward_workspace bytes.
bool fused2_forward_applies(int64_t B, int64_t L, int64_t D, IoType io, const void* x,
                            const void* wr, const void* wi);
size_t fused2_forward_workspace(int64_t B, int64_t L, int64_t D, IoType io);
// With conv taps (w4 [4][D] and b4 [D], as launch_pack_conv packs them; gated
// only) x is hx and x' = SiLU(conv(hx)) is formed on load.
hipError_t launch_fused2_forward(const void* x, const void* wr, const void* br, const void* wi,
                                 const void* bi, const float* lambda, const float* h0, void* h,
                                 float* hT, const void* hz, void* y, int64_t B, int64_t L,
                                 int64_t D, IoType io, void* ws, hipStream_t stream,
                                 const float* w4 = nullptr, const float* b4 = nullptr);

// Scan-algorithm variants for the efficiency ablation (zero initial state;
// x, z, h share the I/O type): a serial scan (one wave per 64 channels walks
// the sequence) and the two-tree scan over the power of two >= L with the
// leading positions as identity (embedding padding), L <= 4096.
// Layer backward's scan with the gate projections recomputed inside
// (scan_bwd_fused_kernel): x, weights packed by channel group
// (launch_pack_groups), biases (may be null); dx in the I/O type, dz_r and
// dz_i in fp32, [B][L][D].
struct FusedBwdArgs {
    const void* x;
    const void* pack;
    const void* br;
    const void* bi;
    const float* lambda;
    const float* h0;
    const void* h;
    const void* dh;
    const float* dhT;
    void* dx;
    float* dzr;
    float* dzi;
    float* dlambda;
    float* dh0;
    int64_t B, L, D;
    IoType io;
    void* ws;
    // Output gate of the gated layer (fp32 x only): when gy is set, dh is
    // formed on load as gy SiLU(gz) (fp32) instead of being read (dh is then
    // unused), and, with fp32 h, if gdz is set, the gate input's gradient
    // gy h SiLU'(gz) is stored there (h's layout).  Folding that gradient in
    // for bf16 h measured slower than its own pass (one extra store and load
    // per element in the scan against a 108 us pass at 16 x 16384 x 256).
    const void* gy = nullptr;
    const void* gz = nullptr;
    void* gdz = nullptr;
    // fp32 x with h, gy, gz, the weights (pack: one bf16 plane, packed from
    // bf16 weights) and the biases in bf16: the gated layer's bf16 backward,
    // which keeps x' and the gradients in fp32.
    bool h_bf16 = false;
};
bool fused_backward_applies(int64_t B, int64_t L, int64_t D, IoType io, const void* x,
                            const void* h, const void* pack);
size_t fused_backward_workspace(int64_t B, int64_t L, int64_t D);
hipError_t launch_fused_backward(const FusedBwdArgs& a, hipStream_t stream);

hipError_t launch_scan_forward_serial(const ScanFwdArgs& a, hipStream_t stream);
hipError_t launch_scan_forward_tree(const ScanFwdArgs& a, hipStream_t stream);
bool tree_scan_supported(int64_t L);
// Backward of the same scan variants (h0 = 0, no dL/dh_T, no dh0): the serial
// walk from t = L - 1 down, or the two-tree scan of the reversed sequence;
// then the gate-gradient epilogue and dLambda.  a.ws takes
// scan_backward_method_workspace(B, D) bytes; bf16 I/O uses bf16 z and dz.
size_t scan_backward_method_workspace(int64_t B, int64_t D);
hipError_t launch_scan_backward_method(bool tree, const ScanBwdArgs& a, hipStream_t stream);

// Gated recurrent layer core (Algorithm alg:gated_recurrent: the causal conv
// + SiLU, the BD-LRU and the output gate).
// Conv taps are packed as [kConvTaps][D] (zero past K) plus a [D] bias.
constexpr int kConvTaps = 4;
hipError_t launch_pack_conv(const float* w, const float* b, int K, int64_t D, float* w4,
                            float* b4, hipStream_t stream);
// x' = SiLU(causal depthwise conv(hx)) into xp ([B][L][D]; hx of type io, x'
// of type out_io: the I/O type, or fp32 for a backward).
hipError_t launch_conv_silu(const void* hx, const float* w4, const float* b4, void* xp, int64_t B,
                            int64_t L, int64_t D, IoType io, IoType out_io, hipStream_t stream);
// y = h * SiLU(hz) over n elements.
hipError_t launch_gate_out(const void* h, const void* hz, void* y, int64_t n, IoType io,
                           hipStream_t stream);
// Output gate backward: dh = dy * SiLU(hz) (stored as dh_io; skipped when dh
// is null), dhz = dy * h * SiLU'(hz) (I/O type).
hipError_t launch_gate_backward(const void* dy, const void* hz, const void* h, void* dh,
                                void* dhz, int64_t n, IoType io, IoType dh_io,
                                hipStream_t stream);
// out[c] = sum over r of src[r][c] ([rows][cols] fp32), in a fixed order in
// double; ws: colsum_workspace bytes.
size_t colsum_workspace(int64_t rows, int64_t cols);
hipError_t launch_colsum(const float* src, int64_t rows, int64_t cols, float* out, void* ws,
                         hipStream_t stream);
// bf16 to fp32 copy of n elements.
hipError_t launch_widen(const void* src, float* dst, int64_t n, hipStream_t stream);
// Conv + SiLU backward from dx' (the BD-LRU input gradient, of type dxp_io):
// dhx, and the tap and bias gradients dw ([D][K]) and db ([D], may be null),
// summed over b and t in a fixed order (double).  ws: conv_backward_workspace
// bytes.
size_t conv_backward_workspace(int64_t B, int64_t L, int64_t D);
hipError_t launch_conv_backward(const void* hx, const void* dxp, const float* w4, const float* b4,
                                void* dhx, float* dw, float* db, int K, int64_t B, int64_t L,
                                int64_t D, IoType io, IoType dxp_io, void* ws,
                                hipStream_t stream);
// The scan forward with the projections fused in (fused_forward_applies) on
// x = x', storing y = h * SiLU(hz) (and h if not null).
hipError_t launch_fused_gated_forward(const void* x, const void* hz, const void* pack,
                                      const void* br, const void* bi, const float* lambda,
                                      const float* h0, void* y, void* h, float* hT, int64_t B,
                                      int64_t L, int64_t D, IoType io, void* ws,
                                      hipStream_t stream);

}  // namespace recblr
