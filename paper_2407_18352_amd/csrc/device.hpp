// Device-side view of a tensor-map plan and the address arithmetic every
// kernel shares: sweep point of a row, boundary resolution, element address.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "plan.hpp"

namespace hpacml {

// Kernel-argument copy of a map plan (passed by value).
struct DevMap {
    int32_t rank, n_features, n_targets, pointwise;
    int64_t n_points;
    int64_t count[HPACML_MAX_RANK];    // sweep points per dimension
    int64_t start[HPACML_MAX_RANK];
    int64_t step[HPACML_MAX_RANK];
    int64_t extent[HPACML_MAX_RANK];
    int32_t bnd[HPACML_MAX_RANK];
    int32_t omin[HPACML_MAX_RANK];
    int32_t omax[HPACML_MAX_RANK];
    int32_t same_strides;              // every target has target 0's strides
    int32_t small_counts;              // every count and n_points < 2^31
    const FeatureEntry *feat;          // [n_features], device
    float *const *base;                // [n_targets], device
    const int64_t *stride;             // [n_targets * 4], device
    int64_t stride0[HPACML_MAX_RANK];  // strides of target 0
};

// Sweep point of row b (row-major over the sweep counts).
__device__ __forceinline__ void sweep_point(const DevMap &m, int64_t b, int64_t p[HPACML_MAX_RANK]) {
#pragma unroll
    for (int d = HPACML_MAX_RANK - 1; d >= 0; --d) {
        if (d < m.rank) {
            int64_t q, r;
            if (m.small_counts) {
                uint32_t bb = (uint32_t)b, c = (uint32_t)m.count[d];
                uint32_t qq = bb / c;
                q = qq;
                r = bb - qq * c;
            } else {
                q = b / m.count[d];
                r = b - q * m.count[d];
            }
            p[d] = m.start[d] + r * m.step[d];
            b = q;
        } else {
            p[d] = 0;
        }
    }
}

// True when every feature's access of point p stays inside the arrays, so the
// precomputed interior offsets apply without boundary handling.
__device__ __forceinline__ bool interior(const DevMap &m, const int64_t p[HPACML_MAX_RANK]) {
    bool ok = true;
#pragma unroll
    for (int d = 0; d < HPACML_MAX_RANK; ++d)
        if (d < m.rank)
            ok = ok && (p[d] + m.omin[d] >= 0) && (p[d] + m.omax[d] < m.extent[d]);
    return ok;
}

// Element index of point p in target t (no offset).
__device__ __forceinline__ int64_t point_elem(const DevMap &m, const int64_t p[HPACML_MAX_RANK], int t) {
    int64_t e = 0;
#pragma unroll
    for (int d = 0; d < HPACML_MAX_RANK; ++d)
        if (d < m.rank)
            e += p[d] * (m.same_strides ? m.stride0[d] : m.stride[t * 4 + d]);
    return e;
}

// Element index of feature e at point p with boundary resolution.
__device__ __forceinline__ int64_t resolved_elem(const DevMap &m, const int64_t p[HPACML_MAX_RANK],
                                                 const FeatureEntry &e) {
    int64_t idx = 0;
#pragma unroll
    for (int d = 0; d < HPACML_MAX_RANK; ++d) {
        if (d < m.rank) {
            int64_t q = p[d] + e.off[d];
            const int64_t n = m.extent[d];
            if (m.bnd[d] == HPACML_BND_PERIODIC)
                q = q >= n ? q - n : q;              // off was reduced into [0, n)
            else if (m.bnd[d] == HPACML_BND_CLAMP)
                q = q < 0 ? 0 : (q >= n ? n - 1 : q);
            idx += q * (m.same_strides ? m.stride0[d] : m.stride[e.target * 4 + d]);
        }
    }
    return idx;
}

// Address of feature f of the point at row b, given its sweep point p.
__device__ __forceinline__ const float *feature_ptr(const DevMap &m, const int64_t p[HPACML_MAX_RANK],
                                                    bool inside, int f) {
    const FeatureEntry e = m.feat[f];
    int64_t idx = inside ? point_elem(m, p, e.target) + e.delta : resolved_elem(m, p, e);
    return m.base[e.target] + idx;
}

// Round to bf16 (nearest even, by the hardware conversion) and back to fp32.
__device__ __forceinline__ float round_bf16(float x) {
    __bf16 h = (__bf16)x;
    return (float)h;
}

__host__ DevMap make_devmap(const MapPlan &p, const FeatureEntry *feat_dev, float *const *base_dev,
                            const int64_t *stride_dev);

}  // namespace hpacml
