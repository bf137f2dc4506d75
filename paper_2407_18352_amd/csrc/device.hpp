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

// Load / store of application data through the global address space: a
// pointer fetched from LDS is generic, and a generic (flat) access counts
// against the LDS counter as well, which would serialise a run of gathers.
__device__ __forceinline__ float ldg(const float *p) {
    return *(const __attribute__((address_space(1))) float *)p;
}
__device__ __forceinline__ uint32_t ldg_bits(const float *p) {
    return *(const __attribute__((address_space(1))) uint32_t *)p;
}
__device__ __forceinline__ void stg(float *p, float v) { *(__attribute__((address_space(1))) float *)p = v; }

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

// Element index of feature e at sweep point p, free of divergent branches so
// that a run of gathers issues all its loads before the first wait: the
// interior form (point element + precomputed offset) and the boundary-
// resolved form are both computed and selected per lane.  `pe` is the
// point's element index in target 0 (used when all targets share strides).
__device__ __forceinline__ int64_t gather_elem(const DevMap &m, const int64_t p[HPACML_MAX_RANK], bool inside,
                                               int64_t pe, const FeatureEntry &e) {
    int64_t res = 0, pt = 0;
#pragma unroll
    for (int d = 0; d < HPACML_MAX_RANK; ++d) {
        if (d < m.rank) {
            const int64_t n = m.extent[d];
            const int64_t st = m.same_strides ? m.stride0[d] : m.stride[e.target * 4 + d];
            const int64_t q = p[d] + e.off[d];
            const int64_t qp = q >= n ? q - n : q;                    // off reduced into [0, n)
            const int64_t qc = q < 0 ? 0 : (q >= n ? n - 1 : q);
            const int64_t r = m.bnd[d] == HPACML_BND_PERIODIC ? qp : (m.bnd[d] == HPACML_BND_CLAMP ? qc : q);
            res += r * st;
            pt += p[d] * st;
        }
    }
    const int64_t in = (m.same_strides ? pe : pt) + e.delta;
    return inside ? in : res;
}

// Address of feature f of the point at row b, given its sweep point p.
__device__ __forceinline__ const float *feature_ptr(const DevMap &m, const int64_t p[HPACML_MAX_RANK],
                                                    bool inside, int f) {
    const FeatureEntry e = m.feat[f];
    int64_t idx = inside ? point_elem(m, p, e.target) + e.delta : resolved_elem(m, p, e);
    return m.base[e.target] + idx;
}

// max(x, 0) in one v_max_f32, for x produced by vector ALU arithmetic (not an
// MFMA result: see relu_mfma): such an x is never a signalling NaN, and in
// IEEE mode v_max_f32 returns the other operand for a quiet NaN, so
// max(NaN, 0) = 0 as for fmaxf.  (fmaxf compiles to a quieting v_max_f32
// x, x before the max, twice the cost.)
__device__ __forceinline__ float relu_arith(float x) {
    float r;
    asm("v_max_f32 %0, 0, %1" : "=v"(r) : "v"(x));
    return r;
}

// max(x, 0) for x an MFMA result, as one v_med3_f32(x, 0, +inf) that the
// compiler sees, so it keeps the wait states an MFMA's result needs before the
// vector ALU reads it (inline assembly would bypass that check).  A NaN gives
// 0, as for fmaxf.
__device__ __forceinline__ float relu_mfma(float x) { return __builtin_amdgcn_fmed3f(x, 0.f, __builtin_inff()); }

// Round to bf16 (nearest even, by the hardware conversion) and back to fp32.
__device__ __forceinline__ float round_bf16(float x) {
    __bf16 h = (__bf16)x;
    return (float)h;
}

// 32-bit view of a map for the MFMA and 32-bit collect kernels.  Valid when
// the point count, every sweep count and every element index fit in int32
// and all targets share strides (the common case); maps outside it take the
// general kernels.
// Division by the sweep counts uses precomputed multipliers: for n < 2^31,
// n / d == (n * magic) >> shift with shift = 31 + ceil(log2 d) and
// magic = ceil(2^shift / d).
struct Map32 {
    int32_t rank, n_features, n_targets, n_points;
    int32_t count[HPACML_MAX_RANK], start[HPACML_MAX_RANK], step[HPACML_MAX_RANK];
    int32_t extent[HPACML_MAX_RANK], stride[HPACML_MAX_RANK];
    int32_t bnd[HPACML_MAX_RANK], omin[HPACML_MAX_RANK], omax[HPACML_MAX_RANK];
    uint32_t magic[HPACML_MAX_RANK];
    int32_t shift[HPACML_MAX_RANK];
};

// A sweep point resolved for gathering: coordinates and element index in
// the (shared) strides.
struct Pt32 {
    int32_t p[HPACML_MAX_RANK];
    int32_t pe;
};

__device__ __forceinline__ Pt32 locate32(const Map32 &m, int32_t b) {
    Pt32 r;
    uint32_t rem = (uint32_t)b;
    r.pe = 0;
#pragma unroll
    for (int d = HPACML_MAX_RANK - 1; d >= 0; --d) {
        if (d < m.rank) {
            const uint32_t q = (uint32_t)(((uint64_t)rem * m.magic[d]) >> m.shift[d]);
            const int32_t k = (int32_t)(rem - q * (uint32_t)m.count[d]);
            rem = q;
            const int32_t x = m.start[d] + k * m.step[d];
            r.p[d] = x;
            r.pe += x * m.stride[d];
        } else {
            r.p[d] = 0;
        }
    }
    return r;
}

// Dimensions along which some lane of the wave reads outside the arrays:
// bit d set when any lane's window leaves [0, extent) along d (wave-uniform).
__device__ __forceinline__ uint32_t edge_dims32(const Map32 &m, const Pt32 &r) {
    uint32_t edge = 0;
#pragma unroll
    for (int d = 0; d < HPACML_MAX_RANK; ++d)
        if (d < m.rank && __any(r.p[d] + m.omin[d] < 0 || r.p[d] + m.omax[d] >= m.extent[d]))
            edge |= 1u << d;
    return edge;
}

// Boundary correction of a feature with raw offsets `raw8` at point r, for
// maps with Map32::raw8: the element index of the access is the interior
// index (point + offset) plus this.  Only the dimensions in the wave-uniform
// set `edge` are resolved (elsewhere every lane is inside and the correction
// is zero): periodic wraps once (|offset| <= extent), clamp saturates.
__device__ __forceinline__ int32_t edge_fix32(const Map32 &m, const Pt32 &r, uint32_t raw8, uint32_t edge) {
    int32_t fix = 0;
#pragma unroll
    for (int d = 0; d < HPACML_MAX_RANK; ++d) {
        if (edge & (1u << d)) {
            const int32_t q = r.p[d] + (int32_t)(int8_t)(raw8 >> (8 * d));
            const int32_t n = m.extent[d];
            int32_t c;
            if (m.bnd[d] == HPACML_BND_PERIODIC)
                c = (n & (q >> 31)) - (n & ~((q - n) >> 31));   // +n below 0, -n at or past n
            else
                c = max(0, min(q, n - 1)) - q;
            fix += c * m.stride[d];
        }
    }
    return fix;
}

// Per-block LDS copy of the parts of a plan that the gathers index with a
// wave-uniform feature number: read from LDS they cost no vector-memory
// counter slots, so the data loads that follow can all be in flight at once.
template <int NF, int NT>
struct LdsPlan {
    FeatureEntry feat[NF];
    float *base[NT];
    // cooperative copy by the whole block; call __syncthreads() after
    template <typename M>
    __device__ void stage(const M &m) {
        for (int i = threadIdx.x; i < m.n_features && i < NF; i += blockDim.x)
            feat[i] = m.feat[i];
        for (int i = threadIdx.x; i < m.n_targets && i < NT; i += blockDim.x)
            base[i] = m.base[i];
    }
};

__host__ DevMap make_devmap(const MapPlan &p, const FeatureEntry *feat_dev, float *const *base_dev,
                            const int64_t *stride_dev);
// Fills `out` and returns true when the map fits the 32-bit view.
__host__ bool make_map32(const MapPlan &p, Map32 *out);

}  // namespace hpacml
