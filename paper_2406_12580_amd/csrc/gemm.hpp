// Host launchers of the gate-projection products (internal to librecblr.so).
#pragma once

#include <initializer_list>

#include "launch.hpp"

namespace recblr {

// Bytes of the packed-weight scratch that launch_project_forward and
// launch_project_backward_data take (16-byte aligned).
size_t project_pack_workspace(int64_t D, IoType io);

// z_r = x W_r^T + b_r, z_i = x W_i^T + b_i over M = B*L rows (b may be null).
// x, W, b and dx use the I/O type; z and dz are always fp32.  The fast path
// needs zi, dzi after zr, dzr in one allocation (their byte distance is used
// as an offset from zr, dzr).
hipError_t launch_project_forward(const void* x, const void* wr, const void* br, const void* wi,
                                  const void* bi, void* zr, void* zi, int64_t M, int64_t D,
                                  IoType io, void* pack, hipStream_t stream);

// dx += dz_r W_r + dz_i W_i (dx holds the direct term on entry); dx is in the
// I/O type, or fp32 when dx_f32 is set.
hipError_t launch_project_backward_data(const void* dzr, const void* dzi, const void* wr,
                                        const void* wi, void* dx, int64_t M, int64_t D,
                                        IoType io, void* pack, hipStream_t stream,
                                        bool dx_f32 = false);

// dW_r, dW_i = dz^T x and db_r, db_i = column sums of dz; uses
// project_dw_workspace(M, D) bytes of scratch at `ws`.
hipError_t launch_project_backward_weights(const void* dzr, const void* dzi, const void* x,
                                           float* dwr, float* dbr, float* dwi, float* dbi,
                                           int64_t M, int64_t D, IoType io, void* ws,
                                           hipStream_t stream);

// Packs [W_r; W_i] by channel group of 64 (rows 128 g.. : W_r rows of the
// group's channels, then their W_i rows) into project_pack_workspace(D, io)
// bytes of bf16 planes, for the scan forward with the projections fused in.
hipError_t launch_pack_groups(const void* wr, const void* wi, int64_t D, IoType io, void* pack,
                              hipStream_t stream);

// Recurrent step with the gate projections fused in (z stays in registers):
// h_next = alpha h_prev + beta x with z = x W^T + b.  Returns false, having
// launched nothing, where the fused path does not apply (D % 8 != 0, x or
// pack not 16-byte aligned, or x too large); else launches and stores the
// launch status in *err.  pack takes step_pack_workspace(D, io) bytes.
size_t step_pack_workspace(int64_t D, IoType io);
bool launch_fused_step(const void* x, const void* wr, const void* br, const void* wi,
                       const void* bi, const float* lambda, const float* h_prev, float* h_next,
                       int64_t B, int64_t D, IoType io, void* pack, hipStream_t stream,
                       hipError_t* err);

// Plain fp32 linear layer Y = X W^T + b, W[N][K] (nn.Linear layout), all
// operands row-major and contiguous, on fp32 matrix-core tiles (fp32
// products): the forward Y[M][N] = X[M][K] W^T + bias (bias may be null;
// act, if given, receives SiLU(Y)), and the data gradient
// dX[M][K] = dY[M][N] W in one of three epilogues: store, accumulate, or
// multiply by SiLU'(aux) with aux[M][K] the SiLU's input.  The data gradient
// first writes W^T into wt (N * K floats).  Preconditions: wgrad_fast_ok for
// the operands and the shape (N and K multiples of 4).
enum class LinearMode { kStore, kAccumulate, kSiluGrad };
hipError_t launch_linear_fwd32(const float* x, const float* w, const float* bias, float* y,
                               float* act, int64_t M, int64_t N, int64_t K, hipStream_t stream);
hipError_t launch_linear_dgrad32(const float* dy, const float* w, float* dx, LinearMode mode,
                                 const float* aux, int64_t M, int64_t N, int64_t K, float* wt,
                                 hipStream_t stream);

// Weight gradient of a plain fp32 linear layer Y = X W^T + b (W[N][K]) on
// the matrix-core tiles (3-term bf16 split of both operands):
// dW[N][K] = dY[M][N]^T X[M][K] and db[N] = column sums of dY (db may be
// null), as split-M partials (wgrad_workspace bytes at ws) summed in a fixed
// order (launch_colsum, colsum_workspace(wgrad_splits, N * K) bytes at
// colsum_ws).  Applies when wgrad_fast_ok holds (row-major contiguous
// operands, N and K multiples of 4, 16-byte alignment, under 2 GiB each).
bool wgrad_fast_ok(std::initializer_list<const void*> ptrs, int64_t M, int64_t N, int64_t K);
int64_t wgrad_splits(int64_t M, int64_t N, int64_t K);
size_t wgrad_workspace(int64_t M, int64_t N, int64_t K);
hipError_t launch_wgrad(const float* dy, const float* x, float* dw, float* db, int64_t M,
                        int64_t N, int64_t K, void* ws, void* colsum_ws, hipStream_t stream);

int64_t project_dw_splits(int64_t M, int64_t D);
size_t project_dw_workspace(int64_t M, int64_t D);

}  // namespace recblr
