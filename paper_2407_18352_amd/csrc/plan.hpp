// Host-side access plan of a tensor map (HIP-free: builds and runs on any CPU).
//
// The paper's data bridge turns a functor applied to a concrete sweep into
// views of application memory in four steps (Sec. IV-A): extraction (offset
// of each slice relative to the sweep point), resolution (element counts per
// dimension), wrapping (views over the application arrays) and composition
// (flatten + concatenate into the feature dimension).  The first three depend
// only on the descriptors, so they are done here once per map; the result is a
// per-feature table that the device kernels index directly, which makes
// composition a gather inside the fused kernel.
#pragma once

#include <cstdint>
#include <vector>

#include "hpacml.h"

namespace hpacml {

// One feature of a map, as the kernels read it (32 bytes).
struct FeatureEntry {
    int32_t target;     // which target array
    int32_t off[HPACML_MAX_RANK];  // offset from the sweep point, per dimension;
                                   // periodic dims: reduced into [0, extent)
    uint32_t raw8;      // raw offsets as four signed bytes (dimension d in
                        // bits 8d..8d+7); meaningful when MapPlan::raw8
    int64_t delta;      // element offset of an interior access:
                        // sum_d raw_offset[d] * stride[target][d]
};
static_assert(sizeof(FeatureEntry) == 32, "FeatureEntry layout");

struct MapPlan {
    int32_t rank = 0, dir = 0, n_targets = 0, n_features = 0;
    int64_t n_points = 0;
    int64_t extent[HPACML_MAX_RANK] = {1, 1, 1, 1};
    int64_t start[HPACML_MAX_RANK] = {0, 0, 0, 0};
    int64_t step[HPACML_MAX_RANK] = {1, 1, 1, 1};
    int64_t count[HPACML_MAX_RANK] = {1, 1, 1, 1};   // sweep points per dimension
    int32_t bnd[HPACML_MAX_RANK] = {0, 0, 0, 0};
    int32_t omin[HPACML_MAX_RANK] = {0, 0, 0, 0};    // raw offset range over features
    int32_t omax[HPACML_MAX_RANK] = {0, 0, 0, 0};
    bool pointwise = false;   // every feature reads the sweep point itself
    bool idx32 = false;       // every element index of every target fits in int32
    bool raw8 = false;        // every raw offset fits a signed byte and, along a
                              // periodic dimension, is at most the extent in size
                              // (one wrap resolves it)
    bool record_view = false; // the tensor [points][features], row-major, is
                              // target 0's memory: record element (b, f) is
                              // base[0][b * n_features + f]
    std::vector<void *> base;             // [n_targets]
    std::vector<int64_t> stride;          // [n_targets * 4]
    std::vector<FeatureEntry> feat;       // [n_features]
    std::vector<int32_t> raw;             // [n_features * 4] raw offsets
    std::vector<int64_t> max_elem;        // [n_targets] largest element index
};

// Validates a map description and builds its plan (no device calls).
hpacml_status build_map_plan(const hpacml_functor *f, int32_t dir, const hpacml_array *targets,
                             int32_t n_targets, const hpacml_sweep *sweep, const int32_t *bnd,
                             MapPlan *out);

// Validates a model description (no device calls).
hpacml_status validate_model(int32_t n_layers, const int32_t *dims, const int32_t *act,
                             int32_t compute);

// How the targets of an inference's `in` (TO) and `out` (FROM) maps meet.
enum class Overlap {
    None,       // disjoint, or a `from` target updates a `to` element-for-element
    Snapshot,   // a `from` target may overwrite an input another point still
                // reads: the inputs must be recorded before any output is written
    OutputRace  // two `from` targets may meet (HPACML_E_ALIAS)
};
Overlap classify_overlap(const MapPlan &in, const MapPlan &out);

// True when two targets provably address disjoint elements.
bool disjoint_targets(const MapPlan &a, int ta, const MapPlan &b, int tb);

// ---- convolutional models

// Image shape (rows, columns, channels) at one point of the stack.
struct CnnShape {
    int32_t h, w, c;
};

// A validated convolutional model description (no device state).
struct CnnPlan {
    int32_t in_channels = 0, height = 0, width = 0, n_layers = 0;
    std::vector<hpacml_layer> layers;
    std::vector<CnnShape> shape;   // [n_layers + 1]: input of layer l; [n_layers] = output
    int64_t max_elems = 0;         // largest h * w * c over `shape` (one image)
};
hpacml_status validate_cnn(int32_t in_channels, int32_t height, int32_t width, int32_t n_layers,
                           const hpacml_layer *layers, CnnPlan *out);

}  // namespace hpacml
