// Collect mode: the values a tensor map addresses, copied bit for bit into a
// dense record dst[p * ld + f] (Sec. III-A-2 and Sec. IV-B: the region's
// mapped inputs and outputs are stored for training).
//
// HBM-bound.  Each block owns tiles of WAVES x 64 sweep points.  Phase 1: one
// lane per point walks the features (the feature index is wave-uniform, so
// the plan entry comes through scalar loads) and loads with coalesced reads
// along the sweep; values land in an LDS tile [point][feature].  Phase 2: the
// block writes the tile's record rows as contiguous runs of F words.
#include "kernels.hpp"

namespace hpacml {

namespace {

constexpr int kBatch = 8;

__global__ void __launch_bounds__(256) collect_kernel(DevMap m, uint32_t *__restrict__ dst,
                                                      int64_t ld, int pitch, int64_t n_tiles) {
    extern __shared__ uint32_t tile[];
    __shared__ LdsPlan<HPACML_MAX_FEATURES, HPACML_MAX_TARGETS> plan;
    plan.stage(m);
    __syncthreads();
    const int F = m.n_features;
    const int P = blockDim.x;                  // points per tile (one per thread)
    const int t = threadIdx.x;
    // phase-2 walk: linear element t of the tile is (row t / F, column t % F)
    const int step_r = P / F, step_f = P % F;
    const int r0 = t / F, f0 = t % F;

    for (int64_t tileno = blockIdx.x; tileno < n_tiles; tileno += gridDim.x) {
        const int64_t b0 = tileno * P;
        const int64_t b = b0 + t;
        const bool valid = b < m.n_points;
        int64_t p[HPACML_MAX_RANK];
        sweep_point(m, valid ? b : m.n_points - 1, p);
        const bool inside = interior(m, p);
        const int64_t pe = point_elem(m, p, 0);

        // feature-uniform batches; loads unconditional (feature numbers
        // clamped) so a batch has all its loads in flight at once
        for (int fb = 0; fb < F; fb += kBatch) {
            uint32_t v[kBatch];
#pragma unroll
            for (int k = 0; k < kBatch; ++k) {
                const int f = fb + k < F ? fb + k : F - 1;
                const FeatureEntry e = plan.feat[f];
                v[k] = ldg_bits(plan.base[e.target] + gather_elem(m, p, inside, pe, e));
            }
#pragma unroll
            for (int k = 0; k < kBatch; ++k)
                if (fb + k < F)
                    tile[t * pitch + fb + k] = v[k];
        }
        __syncthreads();

        const int64_t rows = (m.n_points - b0) < P ? (m.n_points - b0) : P;
        int r = r0, f = f0;
        for (int64_t idx = t; idx < rows * F; idx += P) {
            dst[(b0 + r) * ld + f] = tile[r * pitch + f];
            r += step_r;
            f += step_f;
            if (f >= F) {
                f -= F;
                r += 1;
            }
        }
        __syncthreads();
    }
}

}  // namespace

hipError_t launch_collect(const DevMap &m, uint32_t *dst, int64_t ld, hipStream_t stream) {
    if (m.n_points == 0)
        return hipSuccess;
    const int pitch = m.n_features | 1;        // odd pitch: conflict-free phase-1 stores
    // up to 4 waves, LDS tile at most 64 KB
    int waves = 16384 / (64 * pitch);
    waves = waves < 1 ? 1 : (waves > 4 ? 4 : waves);
    const int threads = 64 * waves;
    const size_t lds = (size_t)threads * pitch * sizeof(uint32_t);
    const int64_t n_tiles = (m.n_points + threads - 1) / threads;
    // LDS per block bounds the blocks per CU; 256 CUs
    int per_cu = (int)(65536 / lds);
    per_cu = per_cu < 1 ? 1 : (per_cu > 8 ? 8 : per_cu);
    int64_t grid = 256LL * per_cu;
    if (grid > n_tiles)
        grid = n_tiles;
    hipError_t e = hipFuncSetAttribute((const void *)collect_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(collect_kernel, dim3((unsigned)grid), dim3(threads), lds, stream, m, dst, ld,
                       pitch, n_tiles);
    return hipGetLastError();
}

}  // namespace hpacml
