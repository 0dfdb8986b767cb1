// Full RecBLR model training step (embedding, behaviour-modelling layers,
// prediction, cross entropy) and Adam: internal interface of model.hip,
// called by the C ABI in capi.cpp after argument validation.
#pragma once

#include <hip/hip_runtime.h>
#include <rocblas/rocblas.h>
#include <stddef.h>
#include <stdint.h>

namespace recblr {
namespace model {

struct Dims {
    int64_t B, T, D, E, V, layers;
    int K;
    float eps;
};

// Dropout and padding of one step: drop probability (0: off), Philox key
// (seed, offset), padding id (-1: none).
struct StepOpts {
    float dropout = 0.0f;
    uint64_t seed = 0, offset = 0;
    int pad_id = -1;
};

// Tensors of one behaviour-modelling layer, in parameter order.
enum LayerTensor {
    kWx, kbx, kWz, kbz, kConvW, kConvB, kWr, kbr, kWi, kbi, kLam,
    kWo, kbo, kLn1g, kLn1b, kW1, kb1, kW2, kb2, kLn2g, kLn2b, kLayerTensors
};

constexpr int64_t kMaxLayers = 64;

int64_t tensor_count(const Dims& d);
// Offsets (floats) of every tensor when off is not null; returns the total
// parameter count, each tensor starting at a multiple of 64 floats.
int64_t param_offsets(const Dims& d, int64_t* off);
// Workspace bytes of train_step (0 if the sort's scratch size is unavailable).
size_t workspace_size(const Dims& d);
int train_step(const Dims& d, const StepOpts& o, const float* params, const int* ids,
               const int* targets, float* grads, float* loss, void* ws, rocblas_handle blas,
               hipStream_t stream);
hipError_t adam(float* p, const float* g, float* m1, float* m2, int64_t n, int64_t step, float lr,
                float b1, float b2, float eps, hipStream_t stream);

}  // namespace model
}  // namespace recblr
