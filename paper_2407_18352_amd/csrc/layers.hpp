// Layer-by-layer MLP inference for shapes outside the fused kernels: one
// gather kernel, one hipBLASLt matmul per layer with the bias and the
// activation in its epilogue, one scatter kernel, over chunks of points.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device.hpp"

namespace hpacml {

struct LayersPlan;   // defined in mlp_layers.hip

// Device copies of the weights (rows padded to 16-byte multiples; bf16
// models: rounded to bf16) and biases.  Nothing of the matmul library is
// touched yet.  Returns hipSuccess and *out, or the allocation/copy error.
hipError_t layers_create(int n_layers, const int32_t *dims, const int32_t *act, const float *const *W,
                         const float *const *b, int compute, LayersPlan **out);
void layers_destroy(LayersPlan *p);

// Whether the plan can run n_points points: on first use per chunk size it
// selects (and caches) the library's algorithm for every layer.  Host only;
// allocates no device memory.
bool layers_ready(LayersPlan *p, int64_t n_points);
const char *layers_name(const LayersPlan *p);

// gather -> every layer -> scatter for all points of `in` / `out`, chunk by
// chunk, on `stream`.  The workspace (two activation buffers of one chunk,
// the fp32 output rows and the library's scratch) is allocated on first
// need and grown as needed; calls sharing a plan must not overlap in time.
// Every chunk reads its inputs before it writes its outputs, but later
// chunks read after earlier ones wrote: inferences whose outputs may
// overwrite inputs read a snapshot record instead.
hipError_t layers_infer(LayersPlan *p, const DevMap &in, const DevMap &out, hipStream_t stream);

}  // namespace hpacml
