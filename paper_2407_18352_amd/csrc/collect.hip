// Collect mode: the values a tensor map addresses, copied bit for bit into a
// dense record dst[p * ld + f] (Sec. III-A-2 and Sec. IV-B: the region's
// mapped inputs and outputs are stored for training).
//
// HBM-bound: every point's F values are read once from the application
// arrays and written once to the record.  One block per tile of P sweep
// points (P = 64 x waves, sized so that several blocks share a CU and keep
// enough loads and stores in flight).  Phase 1: one lane per point walks the
// features in batches whose loads are all issued before the first use (the
// feature index is wave-uniform and its plan entry comes from LDS); the
// values land in an LDS tile laid out exactly as the record rows [point][F].
// Phase 2: the tile's rows form one contiguous run of the record when
// ld == F, which the block writes with 16-byte stores; otherwise row by row.
#include <type_traits>

#include "kernels.hpp"

namespace hpacml {

namespace {

constexpr int kBatch = 16;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void stg4(uint32_t *p, u32x4 v) {
    __builtin_nontemporal_store(v, (__attribute__((address_space(1))) u32x4 *)p);
}
__device__ __forceinline__ void stg1(uint32_t *p, uint32_t v) {
    __builtin_nontemporal_store(v, (__attribute__((address_space(1))) uint32_t *)p);
}

// idx / F for idx < 2^16 and F <= 256: with M = ceil(2^24 / F) the error term
// idx * (M * F - 2^24) stays below 2^24, so the quotient is exact.  The
// product idx * M reaches 2^40, hence 64 bits.
__device__ __forceinline__ uint32_t div_small(uint32_t idx, uint32_t magic) {
    return (uint32_t)(((uint64_t)idx * magic) >> 24);
}

template <bool DENSE>
__global__ void __launch_bounds__(256) collect_kernel(DevMap m, uint32_t *__restrict__ dst, int64_t ld,
                                                      uint32_t magic, int64_t n_tiles) {
    extern __shared__ u32x4 tile4[];
    uint32_t *tile = reinterpret_cast<uint32_t *>(tile4);
    __shared__ LdsPlan<HPACML_MAX_FEATURES, HPACML_MAX_TARGETS> plan;
    plan.stage(m);
    __syncthreads();
    const int F = m.n_features;
    const int P = blockDim.x;                  // points per tile (one per thread)
    const int t = threadIdx.x;

    for (int64_t tileno = blockIdx.x; tileno < n_tiles; tileno += gridDim.x) {
        const int64_t b0 = tileno * P;
        const int64_t b = b0 + t;
        const bool valid = b < m.n_points;
        int64_t p[HPACML_MAX_RANK];
        sweep_point(m, valid ? b : m.n_points - 1, p);
        const bool inside = interior(m, p);
        const int64_t pe = point_elem(m, p, 0);
        const bool fast = __all(inside) && m.same_strides;   // no boundary resolution in this wave

        for (int fb = 0; fb < F; fb += kBatch) {
            uint32_t v[kBatch];
            if (fast) {
#pragma unroll
                for (int k = 0; k < kBatch; ++k) {
                    const int f = fb + k < F ? fb + k : F - 1;
                    const FeatureEntry e = plan.feat[f];
                    v[k] = ldg_bits(plan.base[e.target] + pe + e.delta);
                }
            } else {
#pragma unroll
                for (int k = 0; k < kBatch; ++k) {
                    const int f = fb + k < F ? fb + k : F - 1;
                    const FeatureEntry e = plan.feat[f];
                    v[k] = ldg_bits(plan.base[e.target] + gather_elem(m, p, inside, pe, e));
                }
            }
#pragma unroll
            for (int k = 0; k < kBatch; ++k)
                if (fb + k < F)
                    tile[t * F + fb + k] = v[k];
        }
        __syncthreads();

        const int rows = (m.n_points - b0) < P ? (int)(m.n_points - b0) : P;
        const int n = rows * F;                    // words of this tile
        if (DENSE) {
            // rows b0.. are one run starting at dst + b0 * F (16-byte aligned:
            // dst is, and P * F is a multiple of 4)
            uint32_t *run = dst + b0 * F;
            for (int q = t; q < n / 4; q += P)
                stg4(run + 4 * q, tile4[q]);
            for (int i = (n & ~3) + t; i < n; i += P)
                stg1(run + i, tile[i]);
        } else {
            for (int i = t; i < n; i += P) {
                const uint32_t r = div_small((uint32_t)i, magic);
                const uint32_t f = (uint32_t)i - r * (uint32_t)F;
                stg1(dst + (b0 + r) * ld + f, tile[i]);
            }
        }
        __syncthreads();
    }
}

// 32-bit form: Map32 view, feature table in the kernel arguments, one tile
// of U x 64 points per block of one wave (no block loops over tiles), and
// boundary resolution only along the dimensions where the wave touches an
// edge.  Maps with few features take several points per lane (U > 1), so a
// block still moves a few KB and keeps several loads per lane in flight.
// One launch serves one or two maps (a region's input and output records):
// the first jobs[0].n_tiles blocks take map 0, the rest map 1.
//
// Tile order within a job: blocks of one XCD (blockIdx % 8) take a
// contiguous range of tiles (windowed maps share halo lines in that XCD's
// L2; consecutive tiles write consecutive record runs).
constexpr int kP = 64;   // lanes per block (one wave)

// points per lane for a map of F features: about 8 values per lane
int32_t points_per_lane(int F) { return F == 1 ? 8 : F == 2 ? 4 : F <= 4 ? 2 : 1; }

// (inlined once per job so that every field is read straight from the
// kernel arguments: selecting between the two by reference would copy both
// into private memory)
// PTR: the feature table is read through the job's device pointer instead
// of the kernel arguments (the launch decides when)
template <int U, bool PTR>
__device__ __forceinline__ void collect32_tile(const CollectJob32 &J, int32_t k0, u32x4 *tile4) {
    uint32_t *tile = reinterpret_cast<uint32_t *>(tile4);
    const Map32 &m = J.m;
    const FeatTable32 &c = PTR ? *J.tabp : J.tab;
    const int F = m.n_features;
    const int t = threadIdx.x;
    const int32_t n_tiles = J.n_tiles;
    int32_t tileno = k0;
    if (J.xcd) {
        const int32_t xq = n_tiles / 8, xr = n_tiles % 8, xx = k0 % 8;
        tileno = xx * xq + (xx < xr ? xx : xr) + k0 / 8;
    }
    constexpr int P = kP * U;                      // points per tile
    const int32_t b0 = tileno * P;
    // lane t takes the points b0 + t + 64 u
    Pt32 pt[U];
    uint32_t edge[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t b = (int64_t)b0 + u * kP + t;   // b0 < n_points < 2^31; b may pass it
        pt[u] = locate32(m, b < m.n_points ? (int32_t)b : m.n_points - 1);
        edge[u] = edge_dims32(m, pt[u]);
    }

    if (U == 1) {
        // batches of K features: table entries fb..fb+K-1 exist (fb + K <= 64)
        auto batch = [&](int fb, auto kb) {
            constexpr int K = decltype(kb)::value;
            uint32_t v[K];
            if (edge[0] == 0) {
#pragma unroll
                for (int e = 0; e < K; ++e)
                    v[e] = ldg_bits(c.fptr[fb + e] + pt[0].pe);
            } else {
#pragma unroll
                for (int e = 0; e < K; ++e)
                    v[e] = ldg_bits(c.fptr[fb + e] + (pt[0].pe + edge_fix32(m, pt[0], c.raw8[fb + e], edge[0])));
            }
#pragma unroll
            for (int e = 0; e < K; ++e)
                if (fb + e < F)
                    tile[t * F + fb + e] = v[e];
        };
        int fb = 0;
        for (; fb + 8 <= F; fb += 8)
            batch(fb, std::integral_constant<int, 8>{});
        for (; fb < F; fb += 4)
            batch(fb, std::integral_constant<int, 4>{});
    } else {
        // F <= 4: one feature at a time, U points per lane in flight
        for (int f = 0; f < F; ++f) {
            uint32_t v[U];
#pragma unroll
            for (int u = 0; u < U; ++u)
                v[u] = ldg_bits(c.fptr[f] +
                                (edge[u] ? pt[u].pe + edge_fix32(m, pt[u], c.raw8[f], edge[u]) : pt[u].pe));
#pragma unroll
            for (int u = 0; u < U; ++u)
                tile[(u * kP + t) * F + f] = v[u];
        }
    }
    __syncthreads();

    const int rows = (m.n_points - b0) < P ? (m.n_points - b0) : P;
    const int n = rows * F;                        // words of this tile
    if (J.fs && !J.dense) {
        // feature-major: 64 consecutive points of one feature per store wave
        for (int r = t; r < rows; r += kP)
            for (int f = 0; f < F; ++f)
                stg1(J.dst + (int64_t)f * J.fs + b0 + r, tile[r * F + f]);
    } else if (J.dense) {
        uint32_t *run = J.dst + (int64_t)b0 * F;   // 16-byte aligned: dst is, P * F is a multiple of 4
        for (int q = t; q < n / 4; q += kP)
            stg4(run + 4 * q, tile4[q]);
        for (int i = (n & ~3) + t; i < n; i += kP)
            stg1(run + i, tile[i]);
    } else {
        for (int i = t; i < n; i += kP) {
            const uint32_t r = div_small((uint32_t)i, J.magic);
            const uint32_t f = (uint32_t)i - r * (uint32_t)F;
            stg1(J.dst + ((int64_t)b0 + r) * J.ld + f, tile[i]);
        }
    }
}

template <bool PTR>
__device__ __forceinline__ void collect32_job_tile(const CollectJob32 &J, int32_t k0, u32x4 *tile4) {
    switch (J.ppl) {
    case 8:
        collect32_tile<8, PTR>(J, k0, tile4);
        break;
    case 4:
        collect32_tile<4, PTR>(J, k0, tile4);
        break;
    case 2:
        collect32_tile<2, PTR>(J, k0, tile4);
        break;
    default:
        collect32_tile<1, PTR>(J, k0, tile4);
        break;
    }
}

template <bool PTR>
__global__ void __launch_bounds__(kP) collect32_kernel(CollectJob32 j0, CollectJob32 j1) {
    extern __shared__ u32x4 tile4[];
    if ((int32_t)blockIdx.x < j0.n_tiles)
        collect32_job_tile<PTR>(j0, (int32_t)blockIdx.x, tile4);
    else
        collect32_job_tile<PTR>(j1, (int32_t)blockIdx.x - j0.n_tiles, tile4);
}

}  // namespace

CollectJob32 collect32_job(const MapPlan &p, const Map32 &m, const FeatTable32 &tab, const FeatTable32 *tab_dev,
                           uint32_t *dst, int64_t ld) {
    CollectJob32 j{};
    j.m = m;
    j.tab = tab;
    j.tabp = tab_dev;
    j.dst = dst;
    j.ld = ld;
    const int F = p.n_features;
    j.magic = (uint32_t)(((1u << 24) + F - 1) / F);
    j.ppl = points_per_lane(F);
    j.n_tiles = (int32_t)((p.n_points + (int64_t)kP * j.ppl - 1) / ((int64_t)kP * j.ppl));
    j.dense = ld == F && ((uintptr_t)dst & 15u) == 0;
    j.xcd = !p.pointwise;
    j.fs = 0;
    return j;
}

hipError_t launch_collect32(const CollectJob32 *jobs, int n_jobs, hipStream_t stream) {
    // one launch saves a dispatch (several microseconds) where that matters;
    // large jobs run as separate launches so each gets an LDS tile sized for
    // its own feature count
    constexpr int32_t kFuseMaxTiles = 1 << 17;
    if (n_jobs > 1 && (jobs[0].n_tiles > kFuseMaxTiles || jobs[1].n_tiles > kFuseMaxTiles)) {
        hipError_t e = launch_collect32(jobs, 1, stream);
        return e == hipSuccess ? launch_collect32(jobs + 1, 1, stream) : e;
    }
    CollectJob32 j0 = jobs[0], j1{};
    if (n_jobs > 1)
        j1 = jobs[1];
    else
        j1.n_tiles = 0;
    const int64_t grid = (int64_t)j0.n_tiles + j1.n_tiles;
    if (grid == 0)
        return hipSuccess;
    // LDS tile: the larger of the two jobs' U x 64 x F words
    const int w0 = j0.ppl * j0.m.n_features, w1 = j1.n_tiles ? j1.ppl * j1.m.n_features : 0;
    const size_t lds = (size_t)kP * (w0 > w1 ? w0 : w1) * sizeof(uint32_t);
    // the table through its device pointer when the widest map has 5-16
    // features (one point per lane) and the launch at most 2 x 2^17 tiles
    // (measured: 6-13% faster for the 6- and 9-feature pointwise records;
    // slower for maps of 1-4 features, several points per lane, for the
    // wide windows and on a 2-million-tile launch)
    const int fw = j1.n_tiles && j1.m.n_features > j0.m.n_features ? j1.m.n_features : j0.m.n_features;
    if (fw >= 5 && fw <= 16 && grid <= 2 * kFuseMaxTiles)
        hipLaunchKernelGGL(collect32_kernel<true>, dim3((unsigned)grid), dim3(kP), lds, stream, j0, j1);
    else
        hipLaunchKernelGGL(collect32_kernel<false>, dim3((unsigned)grid), dim3(kP), lds, stream, j0, j1);
    return hipGetLastError();
}

hipError_t launch_collect(const DevMap &m, uint32_t *dst, int64_t ld, hipStream_t stream) {
    if (m.n_points == 0)
        return hipSuccess;
    const int F = m.n_features;
    // tile of P = 64 x waves points, its LDS at most ~40 KB (four or more
    // blocks per CU)
    int waves = 40960 / (256 * F);
    waves = waves < 1 ? 1 : (waves > 4 ? 4 : waves);
    const int threads = 64 * waves;
    const size_t lds = (size_t)threads * F * sizeof(uint32_t);
    const int64_t n_tiles = (m.n_points + threads - 1) / threads;
    const int64_t grid = n_tiles < 0x7FFFFFFF ? n_tiles : 0x7FFFFFFF;
    const uint32_t magic = (uint32_t)(((1u << 24) + F - 1) / F);
    const bool dense = ld == F && ((uintptr_t)dst & 15u) == 0;
    auto kern = dense ? collect_kernel<true> : collect_kernel<false>;
    hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(threads), lds, stream, m, dst, ld, magic, n_tiles);
    return hipGetLastError();
}

}  // namespace hpacml
