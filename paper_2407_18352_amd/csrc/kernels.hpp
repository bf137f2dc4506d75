// Kernel launchers of the library (one per kernel family).  Every launcher
// enqueues on `stream` and returns the HIP launch status.
#pragma once

#include <hip/hip_runtime.h>

#include <cstring>
#include <vector>

#include "device.hpp"

namespace hpacml {

// Plain fp32 [out][in] weights + fp32 biases (bf16 models: values already
// rounded to bf16), used by the general-shape kernel.
struct DevModel {
    int32_t n_layers;
    int32_t bf16;
    int32_t max_width;
    int32_t dims[HPACML_MAX_LAYERS + 1];
    int32_t act[HPACML_MAX_LAYERS];
    const float *W[HPACML_MAX_LAYERS];
    const float *b[HPACML_MAX_LAYERS];
};

// Collect: dst[p * ld + f] = bits of feature f at point p.
hipError_t launch_collect(const DevMap &m, uint32_t *dst, int64_t ld, hipStream_t stream);

// Feature table of a map, passed by value to the 32-bit kernels (kernel
// arguments are read through the scalar cache, so a wave-uniform feature
// number costs no vector instruction): maps with a Map32 view, Map32::raw8
// and at most 64 features.  Entries past the last feature repeat it, so
// batches may read the table unconditionally.
constexpr int kTableMaxF = 64;
struct FeatTable32 {
    const float *fptr[kTableMaxF];  // target base + interior offset of feature f
    uint32_t raw8[kTableMaxF];      // raw offsets, signed bytes
};
bool table32_supported(const MapPlan &p, bool map32);
void table32_make(const MapPlan &p, FeatTable32 *out);
// One map's part of a 32-bit collect launch (kernel argument).
struct CollectJob32 {
    Map32 m;
    FeatTable32 tab;
    const FeatTable32 *tabp;   // device copy of tab (read instead of tab by launches of few features)
    uint32_t *dst;
    int64_t ld;
    uint32_t magic;      // idx / F by multiply-shift (idx < 2^16)
    int32_t n_tiles;     // tiles of ppl x 64 points
    int32_t dense;       // ld == F and a 16-byte aligned record: one contiguous run per tile
    int32_t xcd;         // XCD-contiguous tile order (maps with windows)
    int32_t ppl;         // points per lane: 8, 4, 2 or 1 (F = 1, 2, 3-4, more)
    int64_t fs;          // 0: dst[p * ld + f]; else feature-major dst[f * fs + p] (ld unused)
};
CollectJob32 collect32_job(const MapPlan &p, const Map32 &m, const FeatTable32 &tab, const FeatTable32 *tab_dev,
                           uint32_t *dst, int64_t ld);
// One launch for one or two jobs (n_jobs in {1, 2}).
hipError_t launch_collect32(const CollectJob32 *jobs, int n_jobs, hipStream_t stream);

// General-shape fused gather -> MLP -> scatter (VALU, any widths).
hipError_t launch_mlp_generic(const DevMap &in, const DevMap &out, const DevModel &mdl,
                              hipStream_t stream);

// fp32 register-resident fused kernel: hidden layers of one width H in
// {64, 128}, all weights resident in LDS, MFMA 32x32x2 f32.
struct F32Packed {
    int32_t hid;          // H
    int32_t n_hidden;     // hidden-to-hidden layers (H x H), 0..6
    int32_t ks1;          // K-steps of the first layer (ceil(F_in / 2))
    int32_t f_out;        // outputs (1..8)
    int32_t act[HPACML_MAX_LAYERS];
    int32_t lds_bytes;    // size of the packed image (bytes)
    const float *image;   // device copy of the LDS image
};
bool f32_fast_supported(int n_layers, const int32_t *dims, int compute);
size_t f32_image_floats(int n_layers, const int32_t *dims);
void f32_pack(int n_layers, const int32_t *dims, const float *const *W, const float *const *b,
              float *image);
hipError_t launch_mlp_f32(const Map32 &in, const Map32 &out, const FeatTable32 &tin, const FeatTable32 &tout,
                          const F32Packed &pk, hipStream_t stream);
const char *f32_variant_name(const F32Packed &pk);

// bf16 fused kernel: hidden layers of one width H in {256, 512}; activations
// in LDS, weights streamed from L2 as prepacked MFMA fragments.
struct BF16Packed {
    int32_t hid;          // H
    int32_t n_hidden;     // hidden-to-hidden layers (H x H)
    int32_t ks1;          // 16-wide K-steps of the first layer (F_in <= 64)
    int32_t f_out;        // outputs (1..16)
    int32_t act[HPACML_MAX_LAYERS];
    int64_t off_w1, off_wh, off_wo;   // fragment offsets, 16-byte units
    uint32_t frag_bytes;  // size of the packed fragments
    const void *frags;    // device: packed bf16 fragments (biases folded in)
    float bias_out[16];
};
bool bf16_fast_supported(int n_layers, const int32_t *dims, int compute);
size_t bf16_pack(int n_layers, const int32_t *dims, const float *const *W, const float *const *b,
                 std::vector<uint16_t> &frags, BF16Packed *pk);
hipError_t launch_mlp_bf16(const Map32 &in, const Map32 &out, const FeatTable32 &tin, const FeatTable32 &tout,
                           const BF16Packed &pk, hipStream_t stream);
const char *bf16_variant_name(const BF16Packed &pk);

// Host bf16 helpers shared by the bf16 packers: round to nearest even (NaN
// stays a quiet NaN), the value of a bf16 pattern, and an fp32 bias split
// exactly into three bf16 terms (hi + mid + lo == b).
uint16_t bf16_rne_host(float x);
float bf16_value(uint16_t h);
void split_bias(float b, uint16_t out[3]);

// bf16 fused kernel with register-resident activations: uniform hidden width
// H in {256, 512} (one hidden layer at 512, up to two at 256), ReLU hidden
// layers, F_in <= 45, F_out <= 8.  Weights stream through an LDS ring.
struct BF16RPacked {
    int32_t hid;          // H
    int32_t n_hidden;     // hidden-to-hidden layers (H x H)
    int32_t ks1;          // 16-wide K-steps of the first layer
    int32_t f_out;        // outputs
    int32_t stages;       // 16 KB ring stages per tile of 256 points
    int32_t act[HPACML_MAX_LAYERS];
    const void *stream;   // device: the weight stream of one tile [stages][16][64 lanes][8 bf16]
    const void *w3;       // device: output-layer fragments [H/32][2][64][8 bf16]
    const float *bias;    // device: hidden biases in the accumulator layout [n_hidden][H/32][2][16]
    float bias_out[16];
};
bool bf16r_supported(int n_layers, const int32_t *dims, const int32_t *act, int compute);
// Packed buffers: stream, then w3, then bias (16-byte aligned parts); the
// offsets of w3 and bias in bytes.
void bf16r_pack(int n_layers, const int32_t *dims, const float *const *W, const float *const *b,
                std::vector<uint8_t> &buf, size_t *off_w3, size_t *off_bias, BF16RPacked *pk);
hipError_t launch_mlp_bf16r(const Map32 &in, const Map32 &out, const FeatTable32 &tin, const FeatTable32 &tout,
                            const BF16RPacked &pk, hipStream_t stream);
const char *bf16r_variant_name(const BF16RPacked &pk);

// The status hpacml_infer would return for these handles, without launching.
hpacml_status infer_status(const hpacml_model *model, const hpacml_map *in, const hpacml_map *out);

}  // namespace hpacml
