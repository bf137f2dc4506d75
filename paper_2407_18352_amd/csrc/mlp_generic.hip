// General-shape fused region kernel: gather -> MLP -> scatter for any layer
// widths (up to the library's 4096), fp32 or bf16 semantics, plain VALU
// arithmetic.
//
// It serves the allocation-free entry point for shapes the MFMA kernels do
// not take (the layer-by-layer path needs a workspace), and is that path's
// fallback.  A block owns a tile of P sweep points (fewer for wider layers:
// two buffers within 128 KB of LDS); the composed input tensor and each
// layer's activations live in LDS ([P][pitch], two buffers), so nothing but
// the mapped arrays and the weights touches global memory.  Per layer, thread (o, p) computes
//   acc = b[o] + sum_i W[o][i] * h[p][i]
// with points fastest across a wave, so a wave reads one weight row
// (broadcast) and P activation rows (odd pitch: no bank conflicts).
#include "kernels.hpp"

namespace hpacml {

namespace {

template <bool BF16>
__global__ void __launch_bounds__(256) mlp_generic_kernel(DevMap in, DevMap out, DevModel mdl,
                                                          int P, int pitch, int64_t n_tiles) {
    extern __shared__ float sm[];
    float *buf0 = sm;
    float *buf1 = sm + (size_t)P * pitch;
    const int tid = threadIdx.x, nt = blockDim.x;
    const int F = in.n_features;
    const int L = mdl.n_layers;

    for (int64_t tileno = blockIdx.x; tileno < n_tiles; tileno += gridDim.x) {
        const int64_t b0 = tileno * P;
        const int np = (int)((in.n_points - b0) < P ? (in.n_points - b0) : P);

        // gather (tensor composition), feature-major so reads coalesce along the sweep
        for (int idx = tid; idx < np * F; idx += nt) {
            const int f = idx / np, pp = idx - f * np;
            int64_t p[HPACML_MAX_RANK];
            sweep_point(in, b0 + pp, p);
            float v = *feature_ptr(in, p, interior(in, p), f);
            buf0[pp * pitch + f] = BF16 ? round_bf16(v) : v;
        }
        __syncthreads();

        float *cur = buf0, *nxt = buf1;
        for (int l = 0; l < L; ++l) {
            const int K = mdl.dims[l], N = mdl.dims[l + 1];
            const float *W = mdl.W[l];
            const float *bias = mdl.b[l];
            const bool relu = mdl.act[l] == HPACML_ACT_RELU;
            const bool round = BF16 && l < L - 1;
            for (int idx = tid; idx < np * N; idx += nt) {
                const int o = idx / np, pp = idx - o * np;
                const float *w = W + (size_t)o * K;
                const float *h = cur + pp * pitch;
                float acc = bias[o];
                for (int i = 0; i < K; ++i)
                    acc = fmaf(w[i], h[i], acc);
                if (relu)
                    acc = acc > 0.f ? acc : 0.f;
                if (round)
                    acc = round_bf16(acc);
                nxt[pp * pitch + o] = acc;
            }
            __syncthreads();
            float *t = cur;
            cur = nxt;
            nxt = t;
        }

        // scatter through the `from` map: output g goes to target g
        const int G = out.n_features;
        for (int idx = tid; idx < np * G; idx += nt) {
            const int g = idx / np, pp = idx - g * np;
            int64_t p[HPACML_MAX_RANK];
            sweep_point(out, b0 + pp, p);
            float *dst = const_cast<float *>(feature_ptr(out, p, interior(out, p), g));
            *dst = cur[pp * pitch + g];
        }
        __syncthreads();
    }
}

}  // namespace

hipError_t launch_mlp_generic(const DevMap &in, const DevMap &out, const DevModel &mdl,
                              hipStream_t stream) {
    if (in.n_points == 0)
        return hipSuccess;
    const int pitch = mdl.max_width | 1;
    int P = 16384 / pitch;            // two buffers of P x pitch floats <= 128 KB
    P = P > 64 ? 64 : (P < 1 ? 1 : P);
    const size_t lds = 2 * (size_t)P * pitch * sizeof(float);
    const int64_t n_tiles = (in.n_points + P - 1) / P;
    int64_t grid = n_tiles < 2048 ? n_tiles : 2048;
    const void *fn = mdl.bf16 ? (const void *)mlp_generic_kernel<true> : (const void *)mlp_generic_kernel<false>;
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess)
        return e;
    if (mdl.bf16)
        hipLaunchKernelGGL(mlp_generic_kernel<true>, dim3((unsigned)grid), dim3(256), lds, stream,
                           in, out, mdl, P, pitch, n_tiles);
    else
        hipLaunchKernelGGL(mlp_generic_kernel<false>, dim3((unsigned)grid), dim3(256), lds, stream,
                           in, out, mdl, P, pitch, n_tiles);
    return hipGetLastError();
}

}  // namespace hpacml
