// Convolutional surrogates (the image-shaped model spaces of Table IV):
// host plan, the layer-by-layer kernels and the fused convolution-stack
// kernel.
#pragma once

#include <vector>

#include "kernels.hpp"

namespace hpacml {

// ---- layer-by-layer path: one kernel per layer over S images ([S][h][w][c]
// tensors in a workspace), then a scatter of the last one.
constexpr int kConvG = 8;           // output channels per convolution thread
struct CnnLayerDev {
    int32_t kind, cin, cout, kh, kw, sh, sw, same, mode, act;
    int32_t h, w, h2, w2;          // input and output image sizes
    // i / w2 == (i * w2_magic) >> w2_shift for i < 2^31 (and likewise h2)
    uint32_t w2_magic, w2_shift, h2_magic, h2_shift;
    const float *W, *b;            // device: convolution weights packed by
                                   // cnn_conv_pack, else the caller's layouts
};
// Sets the division constants of L.w2 and L.h2.
void cnn_layer_divisors(CnnLayerDev &L);
// Convolution weights [cout][cin][kh][kw] -> [ceil(cout / kConvG)][kh][kw][cin]
// [kConvG], zero past cout (appended to `dst`).
void cnn_conv_pack(const float *W, int cout, int cin, int kh, int kw, std::vector<float> &dst);
// `part`: scratch of linear_splits(L, S) * S * cout floats for a fully
// connected layer whose K is split over several blocks (unused otherwise)
constexpr int kLinSplit = 32;
int linear_splits(const CnnLayerDev &L, int64_t S);
hipError_t launch_cnn_layer(const CnnLayerDev &L, const float *in, float *out, int64_t S, float *part,
                            hipStream_t stream);
// A convolution and the max-pool after it in one kernel: pools whose
// windows do not overlap (stride == window).
bool cnn_pool_fusable(const CnnLayerDev &conv, const CnnLayerDev &pool);
hipError_t launch_cnn_conv(const CnnLayerDev &L, const CnnLayerDev *pool, const float *in, float *out, int64_t S,
                           hipStream_t stream);
// The fully connected layers that end a stack in one kernel with the
// scatter: cnn_tail_start gives the first of them (any K, at most 256
// outputs; the rest at most 256 wide, at most kTailLayers of them), or -1.
// launch_cnn_linear_partials runs that first layer's products (raw split-K
// partials, or finished outputs when *splits comes back 1); launch_cnn_tail
// the rest.
constexpr int kTailLayers = 4;
struct CnnTail {
    CnnLayerDev first;
    CnnLayerDev rest[kTailLayers];
    int32_t n_rest;
    int32_t splits;                // 0: src holds the first layer's outputs [S][cout]
    int32_t width;                 // power of two >= every layer's width
};
int cnn_tail_start(const std::vector<CnnLayerDev> &ly);
hipError_t launch_cnn_linear_partials(const CnnLayerDev &L, const float *in, float *out, int64_t S, float *part,
                                      int *splits, hipStream_t stream);
hipError_t launch_cnn_tail(const std::vector<CnnLayerDev> &ly, int start, const float *src, int splits,
                           const DevMap &out, int64_t S, hipStream_t stream);
// src[p * F + g] -> feature g of point p of the (FROM) map
hipError_t launch_scatter_record(const DevMap &m, const float *src, hipStream_t stream);

// ---- fused path: a stack of SAME, stride-1 convolutions of at most 16
// channels in one kernel (gather -> every layer in LDS -> scatter).
constexpr int kCnnFusedMaxLayers = 4;
constexpr int kCnnFusedMaxC = 16;
struct CnnFusedLayer {
    int32_t cin4, cout4;           // channel groups of 4 (zero padded)
    int32_t kh, kw, top, left;     // window; padding rows / columns before
    int32_t act;
    int32_t mode;                  // padding mode of this layer's input
    int32_t woff, boff;            // float offsets of the packed weights / biases
};
struct CnnFused {
    int32_t n_layers = 0, c0 = 0, cout_last = 0, circular = 0;
    CnnFusedLayer L[kCnnFusedMaxLayers]{};
    const float *wts = nullptr;    // device: per layer [cout4][ky][kx][cin4*4][4], then bias [cout4*4]
};
bool cnn_fused_supported(const CnnPlan &p);
// Packs the host weights; `out.wts` is left for the caller to set.
void cnn_fused_pack(const CnnPlan &p, const float *const *W, const float *const *b, std::vector<float> &buf,
                    CnnFused *out);
// Rows per tile (64 columns) for this stack, or 0 when no tile fits in LDS.
int cnn_fused_tile_rows(const CnnFused &f, int32_t H);
// tin, tout: device copies of the maps' feature tables
hipError_t launch_cnn_fused(const Map32 &in, const Map32 &out, const FeatTable32 *tin, const FeatTable32 *tout,
                            const CnnFused &f, int32_t S, int32_t H, int32_t W, hipStream_t stream);

}  // namespace hpacml
