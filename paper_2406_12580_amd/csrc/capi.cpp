// C ABI of librecblr.so (declared in include/recblr.h): argument validation,
// workspace carving and dispatch to the HIP kernels.  Validation runs entirely
// on the host and before any HIP call, so a rejected call has enqueued nothing.
#include "recblr.h"

#include <hip/hip_runtime.h>

#include <initializer_list>
#include <utility>

#include "gemm.hpp"
#include "launch.hpp"
#include "model.hpp"

using namespace recblr;

namespace {

constexpr size_t kWsAlign = 256;
constexpr int64_t kMaxDim = (int64_t)1 << 31;       // each of B, L, D
constexpr int64_t kMaxElems = (int64_t)1 << 40;     // B*L*D
constexpr int64_t kMaxChannels = (int64_t)1 << 36;  // B*D (grid of B*D/64 workgroups)
constexpr int64_t kMaxProjD = 1024;
constexpr int64_t kMaxD = (int64_t)65535 * 64;        // channel groups of the dLambda reduction

inline size_t align_up(size_t v) { return (v + kWsAlign - 1) / kWsAlign * kWsAlign; }

struct Buf {
    const void* p;
    size_t bytes;
};

bool overlaps(Buf a, Buf b) {
    if (!a.p || !b.p || a.bytes == 0 || b.bytes == 0) return false;
    uintptr_t a0 = (uintptr_t)a.p, b0 = (uintptr_t)b.p;
    return a0 < b0 + b.bytes && b0 < a0 + a.bytes;
}

bool aligned(const void* p, size_t a) { return p == nullptr || ((uintptr_t)p % a) == 0; }

// Outputs must not overlap inputs or each other.
bool disjoint(std::initializer_list<Buf> outs, std::initializer_list<Buf> ins) {
    for (auto o = outs.begin(); o != outs.end(); ++o) {
        for (const Buf& i : ins)
            if (overlaps(*o, i)) return false;
        for (auto o2 = o + 1; o2 != outs.end(); ++o2)
            if (overlaps(*o, *o2)) return false;
    }
    return true;
}

int check_dims(int64_t B, int64_t L, int64_t D, int io) {
    if (io != RECBLR_F32 && io != RECBLR_BF16) return RECBLR_ERR_UNSUPPORTED;
    if (B < 0 || L < 0 || D < 0) return RECBLR_ERR_INVALID_ARGUMENT;
    if (B >= kMaxDim || L >= kMaxDim || D > kMaxD) return RECBLR_ERR_UNSUPPORTED;
    if (B * D > kMaxChannels) return RECBLR_ERR_UNSUPPORTED;
    if (B * D > 0 && L > kMaxElems / (B * D)) return RECBLR_ERR_UNSUPPORTED;
    return RECBLR_OK;
}

int check_ws(void* ws, size_t ws_bytes, size_t need) {
    if (need == 0) return RECBLR_OK;
    if (ws == nullptr || ws_bytes < need || !aligned(ws, kWsAlign)) return RECBLR_ERR_WORKSPACE;
    return RECBLR_OK;
}

int status_of(hipError_t e) { return e == hipSuccess ? RECBLR_OK : RECBLR_ERR_HIP; }

IoType io_of(int io) { return io == RECBLR_BF16 ? IoType::kBf16 : IoType::kF32; }

size_t esz(int io) { return io == RECBLR_BF16 ? 2 : 4; }

// ---- workspace layouts of the entry points with gate parameters
struct FullFwdLayout {
    size_t zr, zi, pack, scan, total;
};
// z and dz scratch is fp32 whatever the I/O type; z_i follows z_r (and dz_i
// follows dz_r) in the same workspace, which the projection kernels rely on.
FullFwdLayout full_fwd_layout(int64_t B, int64_t L, int64_t D, int io) {
    size_t zbytes = align_up((size_t)(B * L * D) * sizeof(float));
    FullFwdLayout l;
    l.zr = 0;
    l.zi = zbytes;
    l.pack = 2 * zbytes;
    l.scan = l.pack + align_up(project_pack_workspace(D, io_of(io)));
    // The scan part serves either the scan after the projections or the
    // fused kernel (D % 64 == 0), whichever the call takes.
    const size_t scan = scan_forward_workspace(B, L, D, io_of(io));
    const size_t fused = D % 64 == 0 ? fused_forward_workspace(B, L, D) : 0;
    const size_t fused2 = fused2_forward_workspace(B, L, D, io_of(io));
    size_t need = scan > fused ? scan : fused;
    need = need > fused2 ? need : fused2;
    l.total = l.scan + align_up(need);
    return l;
}

struct FullBwdLayout {
    size_t zr, zi, dzr, dzi, pack, scan, dw, total;
};
FullBwdLayout full_bwd_layout(int64_t B, int64_t L, int64_t D, int io) {
    size_t zbytes = align_up((size_t)(B * L * D) * sizeof(float));
    FullBwdLayout l;
    l.zr = 0;
    l.zi = zbytes;
    l.dzr = 2 * zbytes;
    l.dzi = 3 * zbytes;
    l.pack = 4 * zbytes;
    l.scan = l.pack + align_up(project_pack_workspace(D, io_of(io)));
    // The scan part serves either the scan after the projection or the fused
    // kernel (D % 64 == 0), whichever the call takes.
    const size_t scan = scan_backward_workspace(B, L, D, io_of(io));
    const size_t fused = D % 64 == 0 ? fused_backward_workspace(B, L, D) : 0;
    l.dw = l.scan + align_up(scan > fused ? scan : fused);
    l.total = l.dw + align_up(project_dw_workspace(B * L, D));
    return l;
}

// Gated layer: conv taps and bias, then x' and h scratch for the unfused
// path, then the layout of the entry points with weights.
struct GatedLayout {
    size_t w4, b4, xp, hbuf, full, total;
};
GatedLayout gated_layout(int64_t B, int64_t L, int64_t D, int io) {
    GatedLayout l;
    const size_t n = align_up((size_t)(B * L * D) * esz(io));
    l.w4 = 0;
    l.b4 = align_up((size_t)(kConvTaps * D) * sizeof(float));
    l.xp = l.b4 + align_up((size_t)D * sizeof(float));
    l.hbuf = l.xp + n;
    l.full = l.hbuf + n;
    l.total = l.full + full_fwd_layout(B, L, D, io).total;
    return l;
}

// Gated layer backward.  The BD-LRU part runs in fp32 whatever the I/O type
// (its input gradient dh sums over long horizons in the adjoint, so rounding
// it to bf16 costs more than the bf16 tolerance): conv taps, fp32 x', dh and
// dx', for bf16 I/O fp32 copies of h and of the weights, the conv backward
// partials, then the layout of recblr_bdlru_backward at fp32.
struct GatedBwdLayout {
    size_t w4, b4, xp, dh, dxp, h32, wts, conv, full, total;
};
GatedBwdLayout gated_bwd_layout(int64_t B, int64_t L, int64_t D, int io) {
    GatedBwdLayout l;
    const size_t n32 = align_up((size_t)(B * L * D) * sizeof(float));
    const bool widen = io == RECBLR_BF16;
    l.w4 = 0;
    l.b4 = align_up((size_t)(kConvTaps * D) * sizeof(float));
    l.xp = l.b4 + align_up((size_t)D * sizeof(float));
    l.dh = l.xp + n32;
    l.dxp = l.dh + n32;
    l.h32 = l.dxp + n32;
    l.wts = l.h32 + (widen ? n32 : 0);
    l.conv = l.wts + (widen ? align_up((size_t)(2 * D * D + 2 * D) * sizeof(float)) : 0);
    l.full = l.conv + align_up(conv_backward_workspace(B, L, D));
    l.total = l.full + full_bwd_layout(B, L, D, RECBLR_F32).total;
    return l;
}

// Step: z_r, z_i scratch, then the packed weights.
size_t step_z_bytes(int64_t B, int64_t D) { return align_up((size_t)(B * D) * sizeof(float)); }
size_t step_pack_bytes(int64_t D, int io) {
    const size_t a = project_pack_workspace(D, io_of(io)), b = step_pack_workspace(D, io_of(io));
    return align_up(a > b ? a : b);
}
size_t step_ws(int64_t B, int64_t D, int io) {
    return 2 * step_z_bytes(B, D) + step_pack_bytes(D, io);
}

char* at(void* ws, size_t off) { return (char*)ws + off; }

// The scan backward behind recblr_bdlru_scan_backward(_timed) and
// recblr_bdlru_scan_backward_noalloc.  With `static_ws` the scratch is the
// library's static device buffer of the current device (static_scratch);
// otherwise the caller's ws.  Every argument is validated before anything
// is enqueued.
int scan_backward_impl(const void* x, const void* z_r, const void* z_i, const float* lambda,
                       const float* h0, const void* h, const void* dh, const float* dhT,
                       void* dx, void* dz_r, void* dz_i, float* dlambda, float* dh0, int64_t B,
                       int64_t L, int64_t D, int io, void* ws, size_t ws_bytes, bool static_ws,
                       void* stream, void* ev_begin, void* ev_end) {
    int st = check_dims(B, L, D, io);
    if (st) return st;
    if (D == 0) return RECBLR_OK;
    if (!lambda || !dlambda) return RECBLR_ERR_INVALID_ARGUMENT;
    const size_t n = (size_t)(B * L * D) * esz(io), s = (size_t)(B * D) * 4,
                 dl = (size_t)D * 4;
    if (B > 0 && L > 0 && (!x || !z_r || !z_i || !h || !dh || !dx || !dz_r || !dz_i))
        return RECBLR_ERR_INVALID_ARGUMENT;
    for (const void* p : {x, z_r, z_i, h, dh, (const void*)dx, (const void*)dz_r,
                          (const void*)dz_i})
        if (!aligned(p, esz(io))) return RECBLR_ERR_INVALID_ARGUMENT;
    for (const void* p : {(const void*)lambda, (const void*)h0, (const void*)dhT,
                          (const void*)dlambda, (const void*)dh0})
        if (!aligned(p, 4)) return RECBLR_ERR_INVALID_ARGUMENT;
    if (!disjoint({{dx, n}, {dz_r, n}, {dz_i, n}, {dlambda, dl}, {dh0, s}},
                  {{x, n}, {z_r, n}, {z_i, n}, {lambda, dl}, {h0, s}, {h, n}, {dh, n},
                   {dhT, s}}))
        return RECBLR_ERR_INVALID_ARGUMENT;
    hipStream_t strm = (hipStream_t)stream;
    const size_t need = B > 0 ? scan_backward_workspace(B, L, D, io_of(io)) : 0;
    if (static_ws) {
        if (need > kStaticScratchBytes) return RECBLR_ERR_SCRATCH;
        if (need > 0 && static_scratch(&ws, &ws_bytes) != hipSuccess) return RECBLR_ERR_HIP;
    }
    if (B == 0) return status_of(launch_fill(dlambda, 0.0f, D, strm));
    st = check_ws(ws, ws_bytes, need);
    if (st) return st;
    ScanBwdArgs a{x, z_r, z_i, lambda, h0, h, dh, dhT, dx, dz_r, dz_i, dlambda, dh0,
                  B, L, D, io_of(io), io_of(io), ws, ws_bytes,
                  (hipEvent_t)ev_begin, (hipEvent_t)ev_end};
    return status_of(launch_scan_backward(a, strm));
}

}  // namespace

extern "C" {

const char* recblr_status_string(int status) {
    switch (status) {
        case RECBLR_OK: return "ok";
        case RECBLR_ERR_INVALID_ARGUMENT: return "invalid argument";
        case RECBLR_ERR_UNSUPPORTED: return "unsupported";
        case RECBLR_ERR_WORKSPACE: return "workspace missing, too small or misaligned";
        case RECBLR_ERR_HIP: return "HIP launch failure";
        case RECBLR_ERR_SCRATCH:
            return "problem needs more scratch than the library's static device buffer holds";
        default: return "unknown status";
    }
}

size_t recblr_workspace_size(int op, int64_t B, int64_t L, int64_t D, int io) {
    if (op == RECBLR_OP_STEP) L = 1;
    if (check_dims(B, L, D, io) != RECBLR_OK) return 0;
    switch (op) {
        case RECBLR_OP_SCAN_FORWARD: return scan_forward_workspace(B, L, D, io_of(io));
        case RECBLR_OP_SCAN_BACKWARD: return scan_backward_workspace(B, L, D, io_of(io));
        case RECBLR_OP_FORWARD: return full_fwd_layout(B, L, D, io).total;
        case RECBLR_OP_BACKWARD: return full_bwd_layout(B, L, D, io).total;
        case RECBLR_OP_STEP: return step_ws(B, D, io);
        case RECBLR_OP_GATED_FORWARD: return gated_layout(B, L, D, io).total;
        case RECBLR_OP_GATED_BACKWARD: return gated_bwd_layout(B, L, D, io).total;
        case RECBLR_OP_SCAN_BACKWARD_METHOD: {
            const size_t a = scan_backward_workspace(B, L, D, io_of(io)),
                         b = scan_backward_method_workspace(B, D);
            return a > b ? a : b;
        }
        default: return 0;
    }
}

int recblr_bdlru_scan_forward(const void* x, const void* z_r, const void* z_i,
                              const float* lambda, const float* h0, void* h, float* hT,
                              int64_t B, int64_t L, int64_t D, int io, void* ws,
                              size_t ws_bytes, void* stream) {
    return recblr_bdlru_scan_forward_timed(x, z_r, z_i, lambda, h0, h, hT, B, L, D, io, ws,
                                           ws_bytes, stream, nullptr, nullptr);
}

int recblr_bdlru_scan_forward_timed(const void* x, const void* z_r, const void* z_i,
                                    const float* lambda, const float* h0, void* h, float* hT,
                                    int64_t B, int64_t L, int64_t D, int io, void* ws,
                                    size_t ws_bytes, void* stream, void* ev_begin,
                                    void* ev_end) {
    int st = check_dims(B, L, D, io);
    if (st) return st;
    if (B == 0 || D == 0) return RECBLR_OK;
    const size_t n = (size_t)(B * L * D) * esz(io), s = (size_t)(B * D) * 4;
    if (L > 0 && (!x || !z_r || !z_i || !h)) return RECBLR_ERR_INVALID_ARGUMENT;
    if (!lambda) return RECBLR_ERR_INVALID_ARGUMENT;
    for (const void* p : {x, z_r, z_i, (const void*)h})
        if (!aligned(p, esz(io))) return RECBLR_ERR_INVALID_ARGUMENT;
    for (const void* p : {(const void*)lambda, (const void*)h0, (const void*)hT})
        if (!aligned(p, 4)) return RECBLR_ERR_INVALID_ARGUMENT;
    if (!disjoint({{h, n}, {hT, s}},
                  {{x, n}, {z_r, n}, {z_i, n}, {lambda, (size_t)D * 4}, {h0, s}}))
        return RECBLR_ERR_INVALID_ARGUMENT;
    st = check_ws(ws, ws_bytes, scan_forward_workspace(B, L, D, io_of(io)));
    if (st) return st;
    ScanFwdArgs a{x, z_r, z_i, lambda, h0, h, hT, B, L, D, io_of(io), io_of(io), ws, ws_bytes,
                  (hipEvent_t)ev_begin, (hipEvent_t)ev_end};
    return status_of(launch_scan_forward(a, (hipStream_t)stream));
}

int recblr_scan_forward_method(int method, const void* x, const void* z_r, const void* z_i,
                               const float* lambda, void* h, int64_t B, int64_t L, int64_t D,
                               int io, void* ws, size_t ws_bytes, void* stream) {
    if (method == RECBLR_SCAN_CHUNKED)
        return recblr_bdlru_scan_forward(x, z_r, z_i, lambda, nullptr, h, nullptr, B, L, D, io,
                                         ws, ws_bytes, stream);
    if (method != RECBLR_SCAN_SERIAL && method != RECBLR_SCAN_TREE)
        return RECBLR_ERR_INVALID_ARGUMENT;
    int st = check_dims(B, L, D, io);
    if (st) return st;
    if (method == RECBLR_SCAN_TREE && !tree_scan_supported(L)) return RECBLR_ERR_UNSUPPORTED;
    if (B == 0 || D == 0 || L == 0) return RECBLR_OK;
    const size_t n = (size_t)(B * L * D) * esz(io);
    if (!x || !z_r || !z_i || !h || !lambda) return RECBLR_ERR_INVALID_ARGUMENT;
    for (const void* p : {x, z_r, z_i, (const void*)h})
        if (!aligned(p, esz(io))) return RECBLR_ERR_INVALID_ARGUMENT;
    if (!aligned(lambda, 4)) return RECBLR_ERR_INVALID_ARGUMENT;
    if (!disjoint({{h, n}}, {{x, n}, {z_r, n}, {z_i, n}, {lambda, (size_t)D * 4}}))
        return RECBLR_ERR_INVALID_ARGUMENT;
    ScanFwdArgs a{x, z_r, z_i, lambda, nullptr, h, nullptr, B, L, D, io_of(io), io_of(io),
                  nullptr, 0};
    return status_of(method == RECBLR_SCAN_SERIAL ? launch_scan_forward_serial(a, (hipStream_t)stream)
                                                  : launch_scan_forward_tree(a, (hipStream_t)stream));
}

int recblr_scan_backward_method(int method, const void* x, const void* z_r, const void* z_i,
                                const float* lambda, const void* h, const void* dh, void* dx,
                                void* dz_r, void* dz_i, float* dlambda, int64_t B, int64_t L,
                                int64_t D, int io, void* ws, size_t ws_bytes, void* stream) {
    if (method == RECBLR_SCAN_CHUNKED)
        return recblr_bdlru_scan_backward(x, z_r, z_i, lambda, nullptr, h, dh, nullptr, dx, dz_r,
                                          dz_i, dlambda, nullptr, B, L, D, io, ws, ws_bytes,
                                          stream);
    if (method != RECBLR_SCAN_SERIAL && method != RECBLR_SCAN_TREE)
        return RECBLR_ERR_INVALID_ARGUMENT;
    int st = check_dims(B, L, D, io);
    if (st) return st;
    if (method == RECBLR_SCAN_TREE && !tree_scan_supported(L)) return RECBLR_ERR_UNSUPPORTED;
    if (D == 0) return RECBLR_OK;
    if (!lambda || !dlambda) return RECBLR_ERR_INVALID_ARGUMENT;
    const size_t n = (size_t)(B * L * D) * esz(io), dl = (size_t)D * 4;
    if (B > 0 && L > 0 && (!x || !z_r || !z_i || !h || !dh || !dx || !dz_r || !dz_i))
        return RECBLR_ERR_INVALID_ARGUMENT;
    for (const void* p : {x, z_r, z_i, h, dh, (const void*)dx, (const void*)dz_r,
                          (const void*)dz_i})
        if (!aligned(p, esz(io))) return RECBLR_ERR_INVALID_ARGUMENT;
    if (!aligned(lambda, 4) || !aligned(dlambda, 4)) return RECBLR_ERR_INVALID_ARGUMENT;
    if (!disjoint({{dx, n}, {dz_r, n}, {dz_i, n}, {dlambda, dl}},
                  {{x, n}, {z_r, n}, {z_i, n}, {lambda, dl}, {h, n}, {dh, n}}))
        return RECBLR_ERR_INVALID_ARGUMENT;
    hipStream_t strm = (hipStream_t)stream;
    if (B == 0 || L == 0) return status_of(launch_fill(dlambda, 0.0f, D, strm));
    st = check_ws(ws, ws_bytes, scan_backward_method_workspace(B, D));
    if (st) return st;
    ScanBwdArgs a{x, z_r, z_i, lambda, nullptr, h, dh, nullptr, dx, dz_r, dz_i, dlambda, nullptr,
                  B, L, D, io_of(io), io_of(io), ws, ws_bytes};
    return status_of(launch_scan_backward_method(method == RECBLR_SCAN_TREE, a, strm));
}

int recblr_bdlru_scan_backward(const void* x, const void* z_r, const void* z_i,
                               const float* lambda, const float* h0, const void* h,
                               const void* dh, const float* dhT, void* dx, void* dz_r,
                               void* dz_i, float* dlambda, float* dh0, int64_t B, int64_t L,
                               int64_t D, int io, void* ws, size_t ws_bytes, void* stream) {
    return recblr_bdlru_scan_backward_timed(x, z_r, z_i, lambda, h0, h, dh, dhT, dx, dz_r, dz_i,
                                            dlambda, dh0, B, L, D, io, ws, ws_bytes, stream,
                                            nullptr, nullptr);
}

int recblr_bdlru_scan_backward_timed(const void* x, const void* z_r, const void* z_i,
                                     const float* lambda, const float* h0, const void* h,
                                     const void* dh, const float* dhT, void* dx, void* dz_r,
                                     void* dz_i, float* dlambda, float* dh0, int64_t B,
                                     int64_t L, int64_t D, int io, void* ws, size_t ws_bytes,
                                     void* stream, void* ev_begin, void* ev_end) {
    return scan_backward_impl(x, z_r, z_i, lambda, h0, h, dh, dhT, dx, dz_r, dz_i, dlambda, dh0,
                              B, L, D, io, ws, ws_bytes, false, stream, ev_begin, ev_end);
}

int recblr_bdlru_scan_backward_noalloc(const void* x, const void* z_r, const void* z_i,
                                       const float* lambda, const float* h0, const void* h,
                                       const void* dh, const float* dhT, void* dx, void* dz_r,
                                       void* dz_i, float* dlambda, float* dh0, int64_t B,
                                       int64_t L, int64_t D, int io, void* stream) {
    return scan_backward_impl(x, z_r, z_i, lambda, h0, h, dh, dhT, dx, dz_r, dz_i, dlambda, dh0,
                              B, L, D, io, nullptr, 0, true, stream, nullptr, nullptr);
}

int recblr_bdlru_scan_step(const void* x, const void* z_r, const void* z_i,
                           const float* lambda, const float* h_prev, float* h_next, int64_t B,
                           int64_t D, int io, void* stream) {
    int st = check_dims(B, 1, D, io);
    if (st) return st;
    if (B == 0 || D == 0) return RECBLR_OK;
    if (!x || !z_r || !z_i || !lambda || !h_prev || !h_next) return RECBLR_ERR_INVALID_ARGUMENT;
    for (const void* p : {x, z_r, z_i})
        if (!aligned(p, esz(io))) return RECBLR_ERR_INVALID_ARGUMENT;
    for (const void* p : {(const void*)lambda, (const void*)h_prev, (const void*)h_next})
        if (!aligned(p, 4)) return RECBLR_ERR_INVALID_ARGUMENT;
    const size_t n = (size_t)(B * D) * esz(io), s = (size_t)(B * D) * 4;
    // h_next may be h_prev exactly (in-place update) but must not partly overlap it.
    if (h_next != h_prev && overlaps({h_next, s}, {h_prev, s})) return RECBLR_ERR_INVALID_ARGUMENT;
    if (!disjoint({{h_next, s}}, {{x, n}, {z_r, n}, {z_i, n}, {lambda, (size_t)D * 4}}))
        return RECBLR_ERR_INVALID_ARGUMENT;
    return status_of(launch_scan_step(x, z_r, z_i, lambda, h_prev, h_next, B, D, io_of(io),
                                      io_of(io), (hipStream_t)stream));
}

int recblr_bdlru_forward(const void* x, const void* W_r, const void* b_r, const void* W_i,
                         const void* b_i, const float* lambda, const float* h0, void* h,
                         float* hT, int64_t B, int64_t L, int64_t D, int io, void* ws,
                         size_t ws_bytes, void* stream) {
    int st = check_dims(B, L, D, io);
    if (st) return st;
    if (D > kMaxProjD) return RECBLR_ERR_UNSUPPORTED;
    if (B == 0 || D == 0) return RECBLR_OK;
    if (!lambda || !W_r || !W_i || (L > 0 && (!x || !h))) return RECBLR_ERR_INVALID_ARGUMENT;
    for (const void* p : {x, W_r, W_i, b_r, b_i, (const void*)h})
        if (!aligned(p, esz(io))) return RECBLR_ERR_INVALID_ARGUMENT;
    for (const void* p : {(const void*)lambda, (const void*)h0, (const void*)hT})
        if (!aligned(p, 4)) return RECBLR_ERR_INVALID_ARGUMENT;
    const size_t n = (size_t)(B * L * D) * esz(io), s = (size_t)(B * D) * 4,
                 w = (size_t)(D * D) * esz(io), bb = (size_t)D * esz(io);
    if (!disjoint({{h, n}, {hT, s}}, {{x, n}, {W_r, w}, {W_i, w}, {b_r, bb}, {b_i, bb},
                                      {lambda, (size_t)D * 4}, {h0, s}}))
        return RECBLR_ERR_INVALID_ARGUMENT;
    FullFwdLayout lay = full_fwd_layout(B, L, D, io);
    st = check_ws(ws, ws_bytes, lay.total);
    if (st) return st;
    if (!disjoint({{ws, lay.total}}, {{x, n}, {h, n}, {hT, s}, {lambda, (size_t)D * 4}, {h0, s}}))
        return RECBLR_ERR_INVALID_ARGUMENT;
    hipStream_t strm = (hipStream_t)stream;
    void* zr = at(ws, lay.zr);
    void* zi = at(ws, lay.zi);
    void* pack = at(ws, lay.pack);
    if (L > 0 && fused2_forward_applies(B, L, D, io_of(io), x, W_r, W_i))
        return status_of(launch_fused2_forward(x, W_r, b_r, W_i, b_i, lambda, h0, h, hT, nullptr,
                                               nullptr, B, L, D, io_of(io), at(ws, lay.scan),
                                               strm));
    if (L > 0 && fused_forward_applies(B, L, D, io_of(io), x, pack)) {
        hipError_t e = launch_pack_groups(W_r, W_i, D, io_of(io), pack, strm);
        if (e != hipSuccess) return RECBLR_ERR_HIP;
        return status_of(launch_fused_forward(x, pack, b_r, b_i, lambda, h0, h, hT, B, L, D,
                                              io_of(io), at(ws, lay.scan), strm));
    }
    hipError_t e = launch_project_forward(x, W_r, b_r, W_i, b_i, zr, zi, B * L, D, io_of(io),
                                          pack, strm);
    if (e != hipSuccess) return RECBLR_ERR_HIP;
    ScanFwdArgs a{x, zr, zi, lambda, h0, h, hT, B, L, D, io_of(io), IoType::kF32,
                  at(ws, lay.scan), lay.total - lay.scan};
    return status_of(launch_scan_forward(a, strm));
}

int recblr_gated_forward(const void* hx, const void* hz, const float* conv_w,
                         const float* conv_b, int K, const void* W_r, const void* b_r,
                         const void* W_i, const void* b_i, const float* lambda, const float* h0,
                         void* y, void* h, float* hT, int64_t B, int64_t L, int64_t D, int io,
                         void* ws, size_t ws_bytes, void* stream) {
    int st = check_dims(B, L, D, io);
    if (st) return st;
    if (D > kMaxProjD || K < 1 || K > kConvTaps) return RECBLR_ERR_UNSUPPORTED;
    if (B == 0 || D == 0) return RECBLR_OK;
    if (!lambda || !W_r || !W_i || !conv_w || (L > 0 && (!hx || !hz || !y)))
        return RECBLR_ERR_INVALID_ARGUMENT;
    for (const void* p : {hx, hz, W_r, W_i, b_r, b_i, (const void*)y, (const void*)h})
        if (!aligned(p, esz(io))) return RECBLR_ERR_INVALID_ARGUMENT;
    for (const void* p : {(const void*)lambda, (const void*)h0, (const void*)hT,
                          (const void*)conv_w, (const void*)conv_b})
        if (!aligned(p, 4)) return RECBLR_ERR_INVALID_ARGUMENT;
    const size_t n = (size_t)(B * L * D) * esz(io), s = (size_t)(B * D) * 4,
                 w = (size_t)(D * D) * esz(io), bb = (size_t)D * esz(io), df = (size_t)D * 4;
    if (h && overlaps({h, n}, {y, n})) return RECBLR_ERR_INVALID_ARGUMENT;
    if (!disjoint({{y, n}, {h, n}, {hT, s}},
                  {{hx, n}, {hz, n}, {W_r, w}, {W_i, w}, {b_r, bb}, {b_i, bb}, {lambda, df},
                   {h0, s}, {conv_w, (size_t)(D * K) * 4}, {conv_b, df}}))
        return RECBLR_ERR_INVALID_ARGUMENT;
    const GatedLayout lay = gated_layout(B, L, D, io);
    st = check_ws(ws, ws_bytes, lay.total);
    if (st) return st;
    if (!disjoint({{ws, lay.total}}, {{hx, n}, {hz, n}, {y, n}, {h, n}, {hT, s}, {h0, s}}))
        return RECBLR_ERR_INVALID_ARGUMENT;
    hipStream_t strm = (hipStream_t)stream;
    float* w4 = (float*)at(ws, lay.w4);
    float* b4 = (float*)at(ws, lay.b4);
    if (launch_pack_conv(conv_w, conv_b, K, D, w4, b4, strm) != hipSuccess) return RECBLR_ERR_HIP;
    const FullFwdLayout fl = full_fwd_layout(B, L, D, io);
    char* fws = at(ws, lay.full);
    void* pack = fws + fl.pack;
    void* xp = at(ws, lay.xp);
    // Where the weights-resident fused forward applies, x' = SiLU(conv(hx)) is
    // formed on load, from hx rows staged in LDS (with the three before each
    // tile); elsewhere once, by a streaming kernel.
    if (L > 0 && fused2_forward_applies(B, L, D, io_of(io), hx, W_r, W_i))
        return status_of(launch_fused2_forward(hx, W_r, b_r, W_i, b_i, lambda, h0, h, hT, hz, y,
                                               B, L, D, io_of(io), fws + fl.scan, strm, w4, b4));
    if (launch_conv_silu(hx, w4, b4, xp, B, L, D, io_of(io), io_of(io), strm) != hipSuccess)
        return RECBLR_ERR_HIP;
    if (L > 0 && fused_forward_applies(B, L, D, io_of(io), xp, pack)) {
        if (launch_pack_groups(W_r, W_i, D, io_of(io), pack, strm) != hipSuccess)
            return RECBLR_ERR_HIP;
        return status_of(launch_fused_gated_forward(xp, hz, pack, b_r, b_i, lambda, h0, y, h, hT,
                                                    B, L, D, io_of(io), fws + fl.scan, strm));
    }
    // Otherwise the layer forward on x', then the gate.
    void* hout = h ? h : at(ws, lay.hbuf);
    if (L > 0) {
        hipError_t e = launch_project_forward(xp, W_r, b_r, W_i, b_i, fws + fl.zr, fws + fl.zi,
                                              B * L, D, io_of(io), pack, strm);
        if (e != hipSuccess) return RECBLR_ERR_HIP;
    }
    ScanFwdArgs a{xp, fws + fl.zr, fws + fl.zi, lambda, h0, hout, hT, B, L, D, io_of(io),
                  IoType::kF32, fws + fl.scan, fl.total - fl.scan};
    if (launch_scan_forward(a, strm) != hipSuccess) return RECBLR_ERR_HIP;
    return status_of(launch_gate_out(hout, hz, y, B * L * D, io_of(io), strm));
}

int recblr_gated_backward(const void* hx, const void* hz, const float* conv_w,
                          const float* conv_b, int K, const void* W_r, const void* b_r,
                          const void* W_i, const void* b_i, const float* lambda, const float* h0,
                          const void* h, const void* dy, const float* dhT, void* dhx, void* dhz,
                          float* dconv_w, float* dconv_b, float* dW_r, float* db_r, float* dW_i,
                          float* db_i, float* dlambda, float* dh0, int64_t B, int64_t L,
                          int64_t D, int io, void* ws, size_t ws_bytes, void* stream) {
    int st = check_dims(B, L, D, io);
    if (st) return st;
    if (D > kMaxProjD || K < 1 || K > kConvTaps) return RECBLR_ERR_UNSUPPORTED;
    if (D == 0) return RECBLR_OK;
    if (!lambda || !W_r || !W_i || !conv_w || !dconv_w || !dW_r || !dW_i || !db_r || !db_i ||
        !dlambda)
        return RECBLR_ERR_INVALID_ARGUMENT;
    if (B > 0 && L > 0 && (!hx || !hz || !h || !dy || !dhx || !dhz))
        return RECBLR_ERR_INVALID_ARGUMENT;
    for (const void* p : {hx, hz, W_r, W_i, b_r, b_i, h, dy, (const void*)dhx, (const void*)dhz})
        if (!aligned(p, esz(io))) return RECBLR_ERR_INVALID_ARGUMENT;
    for (const void* p : {(const void*)lambda, (const void*)h0, (const void*)dhT,
                          (const void*)conv_w, (const void*)conv_b, (const void*)dconv_w,
                          (const void*)dconv_b, (const void*)dW_r, (const void*)db_r,
                          (const void*)dW_i, (const void*)db_i, (const void*)dlambda,
                          (const void*)dh0})
        if (!aligned(p, 4)) return RECBLR_ERR_INVALID_ARGUMENT;
    const size_t n = (size_t)(B * L * D) * esz(io), s = (size_t)(B * D) * 4,
                 w = (size_t)(D * D) * esz(io), bb = (size_t)D * esz(io), wf = (size_t)(D * D) * 4,
                 df = (size_t)D * 4, cw = (size_t)(D * K) * 4;
    if (!disjoint({{dhx, n}, {dhz, n}, {dconv_w, cw}, {dconv_b, df}, {dW_r, wf}, {db_r, df},
                   {dW_i, wf}, {db_i, df}, {dlambda, df}, {dh0, s}},
                  {{hx, n}, {hz, n}, {conv_w, cw}, {conv_b, df}, {W_r, w}, {W_i, w}, {b_r, bb},
                   {b_i, bb}, {lambda, df}, {h0, s}, {h, n}, {dy, n}, {dhT, s}}))
        return RECBLR_ERR_INVALID_ARGUMENT;
    hipStream_t strm = (hipStream_t)stream;
    const GatedBwdLayout lay = gated_bwd_layout(B, L, D, io);
    st = check_ws(ws, ws_bytes, lay.total);
    if (st) return st;
    if (!disjoint({{ws, lay.total}},
                  {{hx, n}, {hz, n}, {h, n}, {dy, n}, {dhx, n}, {dhz, n}, {dh0, s}, {dhT, s}}))
        return RECBLR_ERR_INVALID_ARGUMENT;
    if (B == 0 || L == 0) {
        // No steps: every sum is empty, and dh0 = dhT (h_L = h0).
        for (auto pr : {std::make_pair(dconv_w, (int64_t)(D * K)), std::make_pair(dconv_b, D),
                        std::make_pair(dW_r, D * D), std::make_pair(dW_i, D * D),
                        std::make_pair(db_r, D), std::make_pair(db_i, D),
                        std::make_pair(dlambda, D)})
            if (pr.first && launch_fill(pr.first, 0.0f, pr.second, strm) != hipSuccess)
                return RECBLR_ERR_HIP;
        if (dh0 && B > 0) {
            hipError_t e = dhT ? hipMemcpyAsync(dh0, dhT, s, hipMemcpyDeviceToDevice, strm)
                               : launch_fill(dh0, 0.0f, B * D, strm);
            if (e != hipSuccess) return RECBLR_ERR_HIP;
        }
        return RECBLR_OK;
    }
    float* w4 = (float*)at(ws, lay.w4);
    float* b4 = (float*)at(ws, lay.b4);
    void* xp = at(ws, lay.xp);
    void* dh = at(ws, lay.dh);
    void* dxp = at(ws, lay.dxp);
    const int64_t n_el = B * L * D;
    if (launch_pack_conv(conv_w, conv_b, K, D, w4, b4, strm) != hipSuccess) return RECBLR_ERR_HIP;
    if (launch_conv_silu(hx, w4, b4, xp, B, L, D, io_of(io), IoType::kF32, strm) != hipSuccess)
        return RECBLR_ERR_HIP;
    {
        // The output gate folded into the fused scan: dh = dy SiLU(hz) formed
        // in fp32 on load (dh never reaches memory) and, for fp32 I/O,
        // dhz = dy h SiLU'(hz) stored by the same pass.  x' and the gradients
        // stay fp32; for bf16 I/O h, dy, hz are read as stored (x' or dh
        // rounded to bf16 would move dW by up to 1.5% and dhx by 1.3%; h is
        // exact in bf16).
        void* lws = at(ws, lay.full);
        const FullBwdLayout fl = full_bwd_layout(B, L, D, RECBLR_F32);
        void* pack = at(lws, fl.pack);
        if (fused_backward_applies(B, L, D, IoType::kF32, xp, h, pack)) {
            const bool bf = io == RECBLR_BF16;
            void* dzr = at(lws, fl.dzr);
            void* dzi = at(lws, fl.dzi);
            // bf16: dhz = dy h SiLU'(hz) in a pass of its own (reading dy, hz, h
            // as stored), which measured faster than folding it into the scan;
            // the scan recomputes z from fp32 x' with the weights and biases as
            // given (bf16 weights are one exact operand plane).
            if ((bf && launch_gate_backward(dy, hz, h, nullptr, dhz, n_el, IoType::kBf16,
                                            IoType::kBf16, strm) != hipSuccess) ||
                launch_pack_groups(W_r, W_i, D, io_of(io), pack, strm) != hipSuccess)
                return RECBLR_ERR_HIP;
            FusedBwdArgs fa{xp,        pack,      b_r,     b_i,         lambda, h0, h, nullptr,
                            dhT,       dxp,       (float*)dzr, (float*)dzi, dlambda, dh0,
                            B,         L,         D,       IoType::kF32, at(lws, fl.scan)};
            fa.gy = dy;
            fa.gz = hz;
            fa.gdz = bf ? nullptr : dhz;
            fa.h_bf16 = bf;
            if (launch_fused_backward(fa, strm) != hipSuccess) return RECBLR_ERR_HIP;
            // dx' += dz W (for bf16 I/O with the bf16 weights as given: one
            // operand plane), then dW from fp32 x'.
            if (launch_project_backward_data(dzr, dzi, W_r, W_i, dxp, B * L, D,
                                             bf ? IoType::kBf16 : IoType::kF32, pack, strm,
                                             bf) != hipSuccess ||
                launch_project_backward_weights(dzr, dzi, xp, dW_r, db_r, dW_i, db_i, B * L, D,
                                                IoType::kF32, at(lws, fl.dw), strm) != hipSuccess)
                return RECBLR_ERR_HIP;
            return status_of(launch_conv_backward(hx, dxp, w4, b4, dhx, dconv_w, dconv_b, K, B,
                                                  L, D, io_of(io), IoType::kF32, at(ws, lay.conv),
                                                  strm));
        }
    }
    if (launch_gate_backward(dy, hz, h, dh, dhz, n_el, io_of(io), IoType::kF32, strm) !=
        hipSuccess)
        return RECBLR_ERR_HIP;
    // fp32 views of h and of the weights for the BD-LRU backward.
    const void *h32 = h, *wr32 = W_r, *br32 = b_r, *wi32 = W_i, *bi32 = b_i;
    if (io == RECBLR_BF16) {
        float* hw = (float*)at(ws, lay.h32);
        float* wt = (float*)at(ws, lay.wts);
        if (launch_widen(h, hw, n_el, strm) != hipSuccess ||
            launch_widen(W_r, wt, D * D, strm) != hipSuccess ||
            launch_widen(W_i, wt + D * D, D * D, strm) != hipSuccess ||
            (b_r && launch_widen(b_r, wt + 2 * D * D, D, strm) != hipSuccess) ||
            (b_i && launch_widen(b_i, wt + 2 * D * D + D, D, strm) != hipSuccess))
            return RECBLR_ERR_HIP;
        h32 = hw;
        wr32 = wt;
        wi32 = wt + D * D;
        br32 = b_r ? wt + 2 * D * D : nullptr;
        bi32 = b_i ? wt + 2 * D * D + D : nullptr;
    }
    st = recblr_bdlru_backward(xp, wr32, br32, wi32, bi32, lambda, h0, h32, dh, dhT, dxp, dW_r,
                               db_r, dW_i, db_i, dlambda, dh0, B, L, D, RECBLR_F32,
                               at(ws, lay.full), lay.total - lay.full, stream);
    if (st) return st;
    return status_of(launch_conv_backward(hx, dxp, w4, b4, dhx, dconv_w, dconv_b, K, B, L, D,
                                          io_of(io), IoType::kF32, at(ws, lay.conv), strm));
}

int recblr_bdlru_backward(const void* x, const void* W_r, const void* b_r, const void* W_i,
                          const void* b_i, const float* lambda, const float* h0, const void* h,
                          const void* dh, const float* dhT, void* dx, float* dW_r, float* db_r,
                          float* dW_i, float* db_i, float* dlambda, float* dh0, int64_t B,
                          int64_t L, int64_t D, int io, void* ws, size_t ws_bytes,
                          void* stream) {
    int st = check_dims(B, L, D, io);
    if (st) return st;
    if (D > kMaxProjD) return RECBLR_ERR_UNSUPPORTED;
    if (D == 0) return RECBLR_OK;
    if (!lambda || !W_r || !W_i || !dlambda || !dW_r || !dW_i || !db_r || !db_i)
        return RECBLR_ERR_INVALID_ARGUMENT;
    if (B > 0 && L > 0 && (!x || !h || !dh || !dx)) return RECBLR_ERR_INVALID_ARGUMENT;
    for (const void* p : {x, W_r, W_i, b_r, b_i, h, dh, (const void*)dx})
        if (!aligned(p, esz(io))) return RECBLR_ERR_INVALID_ARGUMENT;
    for (const void* p : {(const void*)lambda, (const void*)h0, (const void*)dhT,
                          (const void*)dW_r, (const void*)db_r, (const void*)dW_i,
                          (const void*)db_i, (const void*)dlambda, (const void*)dh0})
        if (!aligned(p, 4)) return RECBLR_ERR_INVALID_ARGUMENT;
    const size_t n = (size_t)(B * L * D) * esz(io), s = (size_t)(B * D) * 4,
                 w = (size_t)(D * D) * esz(io), bb = (size_t)D * esz(io), wf = (size_t)(D * D) * 4,
                 df = (size_t)D * 4;
    if (!disjoint({{dx, n}, {dW_r, wf}, {db_r, df}, {dW_i, wf}, {db_i, df}, {dlambda, df},
                   {dh0, s}},
                  {{x, n}, {W_r, w}, {W_i, w}, {b_r, bb}, {b_i, bb}, {lambda, df}, {h0, s},
                   {h, n}, {dh, n}, {dhT, s}}))
        return RECBLR_ERR_INVALID_ARGUMENT;
    hipStream_t strm = (hipStream_t)stream;
    FullBwdLayout lay = full_bwd_layout(B, L, D, io);
    st = check_ws(ws, ws_bytes, lay.total);
    if (st) return st;
    void* zr = at(ws, lay.zr);
    void* zi = at(ws, lay.zi);
    void* dzr = at(ws, lay.dzr);
    void* dzi = at(ws, lay.dzi);
    hipError_t e = hipSuccess;
    if (B == 0) {
        // Sums over an empty batch: every parameter gradient is zero.
        for (float* p : {dW_r, dW_i})
            if ((e = launch_fill(p, 0.0f, D * D, strm)) != hipSuccess) return RECBLR_ERR_HIP;
        for (float* p : {db_r, db_i, dlambda})
            if ((e = launch_fill(p, 0.0f, D, strm)) != hipSuccess) return RECBLR_ERR_HIP;
        return RECBLR_OK;
    }
    const int64_t M = B * L;
    void* pack = at(ws, lay.pack);
    if (L > 0 && fused_backward_applies(B, L, D, io_of(io), x, h, pack)) {
        // The scan backward recomputes z on the matrix cores (z never reaches HBM).
        if (launch_pack_groups(W_r, W_i, D, io_of(io), pack, strm) != hipSuccess)
            return RECBLR_ERR_HIP;
        const FusedBwdArgs fa{x,  pack, b_r, b_i, lambda, h0, h, dh, dhT, dx, (float*)dzr,
                              (float*)dzi, dlambda, dh0, B, L, D, io_of(io), at(ws, lay.scan)};
        e = launch_fused_backward(fa, strm);
    } else {
        e = launch_project_forward(x, W_r, b_r, W_i, b_i, zr, zi, M, D, io_of(io), pack, strm);
        if (e != hipSuccess) return RECBLR_ERR_HIP;
        ScanBwdArgs a{x, zr, zi, lambda, h0, h, dh, dhT, dx, dzr, dzi, dlambda, dh0,
                      B, L, D, io_of(io), IoType::kF32, at(ws, lay.scan), lay.dw - lay.scan};
        e = launch_scan_backward(a, strm);
    }
    if (e != hipSuccess) return RECBLR_ERR_HIP;
    e = launch_project_backward_data(dzr, dzi, W_r, W_i, dx, M, D, io_of(io), at(ws, lay.pack),
                                     strm);
    if (e != hipSuccess) return RECBLR_ERR_HIP;
    e = launch_project_backward_weights(dzr, dzi, x, dW_r, db_r, dW_i, db_i, M, D, io_of(io),
                                        at(ws, lay.dw), strm);
    return status_of(e);
}

int recblr_bdlru_step(const void* x, const void* W_r, const void* b_r, const void* W_i,
                      const void* b_i, const float* lambda, const float* h_prev, float* h_next,
                      int64_t B, int64_t D, int io, void* ws, size_t ws_bytes, void* stream) {
    int st = check_dims(B, 1, D, io);
    if (st) return st;
    if (D > kMaxProjD) return RECBLR_ERR_UNSUPPORTED;
    if (B == 0 || D == 0) return RECBLR_OK;
    if (!x || !W_r || !W_i || !lambda || !h_prev || !h_next) return RECBLR_ERR_INVALID_ARGUMENT;
    for (const void* p : {x, W_r, W_i, b_r, b_i})
        if (!aligned(p, esz(io))) return RECBLR_ERR_INVALID_ARGUMENT;
    for (const void* p : {(const void*)lambda, (const void*)h_prev, (const void*)h_next})
        if (!aligned(p, 4)) return RECBLR_ERR_INVALID_ARGUMENT;
    const size_t n = (size_t)(B * D) * esz(io), s = (size_t)(B * D) * 4,
                 w = (size_t)(D * D) * esz(io), bb = (size_t)D * esz(io);
    if (h_next != h_prev && overlaps({h_next, s}, {h_prev, s})) return RECBLR_ERR_INVALID_ARGUMENT;
    if (!disjoint({{h_next, s}}, {{x, n}, {W_r, w}, {W_i, w}, {b_r, bb}, {b_i, bb},
                                  {lambda, (size_t)D * 4}}))
        return RECBLR_ERR_INVALID_ARGUMENT;
    const size_t need = step_ws(B, D, io);
    st = check_ws(ws, ws_bytes, need);
    if (st) return st;
    hipStream_t strm = (hipStream_t)stream;
    void* zr = ws;
    void* zi = at(ws, step_z_bytes(B, D));
    void* pack = at(ws, 2 * step_z_bytes(B, D));
    hipError_t e = hipSuccess;
    if (launch_step_resident(x, W_r, b_r, W_i, b_i, lambda, h_prev, h_next, B, D, io_of(io),
                             strm, &e))
        return status_of(e);
    if (launch_fused_step(x, W_r, b_r, W_i, b_i, lambda, h_prev, h_next, B, D, io_of(io), pack,
                          strm, &e))
        return status_of(e);
    e = launch_project_forward(x, W_r, b_r, W_i, b_i, zr, zi, B, D, io_of(io), pack, strm);
    if (e != hipSuccess) return RECBLR_ERR_HIP;
    return status_of(
        launch_scan_step(x, zr, zi, lambda, h_prev, h_next, B, D, io_of(io), IoType::kF32, strm));
}

}  // extern "C"

namespace {
bool model_dims_ok(const recblr_model_dims* m) {
    if (!m) return false;
    const int64_t ED = m->E * m->D;
    return m->B >= 1 && m->T >= 1 && (m->D == 64 || m->D == 128 || m->D == 256) && m->E >= 1 &&
           ED <= kMaxProjD && m->V >= 1 && m->V < (1ll << 31) && m->layers >= 1 &&
           m->layers <= model::kMaxLayers && m->K >= 1 && m->K <= kConvTaps &&
           m->ln_eps >= 0.0f && m->B * m->T < (1ll << 31) && m->B * m->V < (1ll << 31);
}
model::Dims model_dims(const recblr_model_dims* m) {
    return model::Dims{m->B, m->T, m->D, m->E, m->V, m->layers, m->K, m->ln_eps};
}
}  // namespace

extern "C" {

size_t recblr_model_param_count(const recblr_model_dims* m) {
    return model_dims_ok(m) ? (size_t)model::param_offsets(model_dims(m), nullptr) : 0;
}

int64_t recblr_model_param_offsets(const recblr_model_dims* m, int64_t* offsets, int64_t n) {
    if (!model_dims_ok(m)) return -1;
    const model::Dims d = model_dims(m);
    const int64_t count = model::tensor_count(d);
    int64_t all[3 + model::kLayerTensors * model::kMaxLayers];
    model::param_offsets(d, all);
    for (int64_t i = 0; offsets && i < n && i < count; ++i) offsets[i] = all[i];
    return count;
}

size_t recblr_model_workspace_size(const recblr_model_dims* m) {
    return model_dims_ok(m) ? model::workspace_size(model_dims(m)) : 0;
}

int recblr_blas_create(void** handle) {
    if (!handle) return RECBLR_ERR_INVALID_ARGUMENT;
    rocblas_handle h = nullptr;
    if (rocblas_create_handle(&h) != rocblas_status_success) return RECBLR_ERR_HIP;
    *handle = (void*)h;
    return RECBLR_OK;
}

int recblr_blas_destroy(void* handle) {
    if (!handle) return RECBLR_OK;
    return rocblas_destroy_handle((rocblas_handle)handle) == rocblas_status_success
               ? RECBLR_OK
               : RECBLR_ERR_HIP;
}

int recblr_model_train_step(const recblr_model_dims* m, const recblr_model_step_opts* opts,
                            const float* params, const int32_t* ids, const int32_t* targets,
                            float* grads, float* loss, void* ws, size_t ws_bytes, void* blas,
                            void* stream) {
    if (!m) return RECBLR_ERR_INVALID_ARGUMENT;
    if (!model_dims_ok(m)) return RECBLR_ERR_UNSUPPORTED;
    model::StepOpts o;
    if (opts) {
        // NaN fails both comparisons
        if (!(opts->dropout >= 0.0f && opts->dropout < 1.0f) || opts->pad_id < -1 ||
            opts->pad_id >= m->V)
            return RECBLR_ERR_INVALID_ARGUMENT;
        o.dropout = opts->dropout;
        o.seed = opts->seed;
        o.offset = opts->offset;
        o.pad_id = opts->pad_id;
    }
    if (!params || !ids || !targets || !grads || !loss || !blas)
        return RECBLR_ERR_INVALID_ARGUMENT;
    if (!aligned(params, kWsAlign) || !aligned(grads, kWsAlign) || !aligned(ids, 4) ||
        !aligned(targets, 4) || !aligned(loss, 4))
        return RECBLR_ERR_INVALID_ARGUMENT;
    const model::Dims d = model_dims(m);
    const size_t np = (size_t)model::param_offsets(d, nullptr) * 4,
                 ni = (size_t)(m->B * m->T) * 4, nt = (size_t)m->B * 4;
    if (!disjoint({{grads, np}, {loss, 4}}, {{params, np}, {ids, ni}, {targets, nt}}) ||
        overlaps({grads, np}, {loss, 4}))
        return RECBLR_ERR_INVALID_ARGUMENT;
    const size_t need = model::workspace_size(d);
    if (need == 0) return RECBLR_ERR_UNSUPPORTED;
    int st = check_ws(ws, ws_bytes, need);
    if (st) return st;
    if (!disjoint({{ws, need}}, {{params, np}, {ids, ni}, {targets, nt}, {grads, np}, {loss, 4}}))
        return RECBLR_ERR_INVALID_ARGUMENT;
    return model::train_step(d, o, params, ids, targets, grads, loss, ws, (rocblas_handle)blas,
                             (hipStream_t)stream);
}

int recblr_adam_update(float* params, const float* grads, float* m1, float* m2, int64_t n,
                       int64_t step, float lr, float beta1, float beta2, float eps,
                       void* stream) {
    if (n < 0 || step < 1) return RECBLR_ERR_INVALID_ARGUMENT;
    if (n == 0) return RECBLR_OK;
    if (!params || !grads || !m1 || !m2) return RECBLR_ERR_INVALID_ARGUMENT;
    for (const void* p : {(const void*)params, (const void*)grads, (const void*)m1,
                          (const void*)m2})
        if (!aligned(p, 4)) return RECBLR_ERR_INVALID_ARGUMENT;
    const size_t b = (size_t)n * 4;
    if (overlaps({params, b}, {grads, b}) || overlaps({params, b}, {m1, b}) ||
        overlaps({params, b}, {m2, b}) || overlaps({m1, b}, {m2, b}) ||
        overlaps({grads, b}, {m1, b}) || overlaps({grads, b}, {m2, b}))
        return RECBLR_ERR_INVALID_ARGUMENT;
    return status_of(model::adam(params, grads, m1, m2, n, step, lr, beta1, beta2, eps,
                                 (hipStream_t)stream));
}

int recblr_linear_scan_forward(const float* a, const float* u, const float* h0, float* h,
                               float* hT, int64_t B, int64_t L, int64_t D, void* stream) {
    int st = check_dims(B, L, D, RECBLR_F32);
    if (st) return st;
    if (B == 0 || D == 0) return RECBLR_OK;
    if (L > 0 && (!a || !u || !h)) return RECBLR_ERR_INVALID_ARGUMENT;
    for (const void* p : {(const void*)a, (const void*)u, (const void*)h0, (const void*)h,
                          (const void*)hT})
        if (!aligned(p, 4)) return RECBLR_ERR_INVALID_ARGUMENT;
    const size_t n = (size_t)(B * L * D) * 4, s = (size_t)(B * D) * 4;
    if (!disjoint({{h, n}, {hT, s}}, {{a, n}, {u, n}, {h0, s}}))
        return RECBLR_ERR_INVALID_ARGUMENT;
    return status_of(launch_linear_scan(a, u, h0, h, hT, B, L, D, (hipStream_t)stream));
}

}  // extern "C"
