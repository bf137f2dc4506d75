// Convolutional surrogates on the composed tensor seen as images (Table VI
// model spaces: convolutions of a few channels for MiniWeather; convolution,
// max-pool and fully connected layers for ParticleFilter).
//
// Fused path (convolution-only stacks, SAME padding, stride 1, <= 16
// channels): plain fp32 FMA work with small channel counts, so VALU-bound,
// not a contraction worth MFMA tiles (8 output channels would fill a quarter
// of a 32-wide MFMA).  One block owns a tile of TY x 64 output pixels of one
// image.  It gathers the tile plus the stack's total halo through the `to`
// map into LDS ([row][column][channel], channels padded to 4), then runs every
// layer over the shrinking region — each layer's output region is the next
// layer's input region — and the last layer's outputs go straight from
// registers through the `from` map.  One thread computes one pixel's output
// channels per pass: 16-byte LDS reads of its window, weights as wave-uniform
// scalar loads (one FMA per weight per lane), no bank conflicts for 4-channel
// rows.  Outside the image, a layer's input follows its padding mode:
// circular stacks wrap at the gather and then compute the halo as is (on a
// torus the halo's values equal the wrapped ones); zeros writes 0; replicate
// computes the pixel at the clamped position (inside the region, since the
// region always contains the image edge it crosses).
//
// Layer-by-layer path: one kernel per layer over [S][h][w][c] workspaces
// (one thread per output element), then a scatter of the last tensor.
#include "cnn.hpp"

namespace hpacml {

namespace {

constexpr int kThreads = 256;
constexpr int kTX = 64;   // tile columns

// ------------------------------------------------------------------ fused
struct FusedArgs {
    Map32 in, out;
    FeatTable32 tin, tout;
    int32_t S, H, W, n_layers;
    int32_t ty, tiles_x, tiles_y, n_tiles;
    int32_t c0, cout_last, circular, buf1;   // buf1: float offset of the second LDS buffer
    // region of layer l's input (l = n_layers: the tile itself), relative to
    // the tile origin: rows [-rt, ty + rb), columns [-rl, 64 + rr)
    int32_t rt[kCnnFusedMaxLayers + 1], rl[kCnnFusedMaxLayers + 1];
    int32_t rh[kCnnFusedMaxLayers + 1], rw[kCnnFusedMaxLayers + 1];
    CnnFusedLayer L[kCnnFusedMaxLayers];
};

__device__ __forceinline__ int wrap(int v, int n) {
    int r = v % n;
    return r < 0 ? r + n : r;
}

// Layer 0's input region from the `to` map: pixel (y, x) of image s is
// composed point (s * H + y) * W + x; channel f is its feature f.
template <int CI>
__device__ __forceinline__ void gather_region(const FusedArgs &a, int s, int y0, int x0, float *dst) {
    const int rh = a.rh[0], rw = a.rw[0], n = rh * rw;
    const int mode = a.L[0].mode;
    const int vy0 = y0 - a.rt[0], vx0 = x0 - a.rl[0];
    for (int i = threadIdx.x; i < n; i += kThreads) {
        const int ry = i / rw, rx = i - ry * rw;
        int y = vy0 + ry, x = vx0 + rx;
        bool zero = false;
        if (y < 0 || y >= a.H || x < 0 || x >= a.W) {
            if (mode == HPACML_PADMODE_CIRCULAR) {
                y = wrap(y, a.H);
                x = wrap(x, a.W);
            } else {
                zero = mode == HPACML_PADMODE_ZEROS;
                y = min(max(y, 0), a.H - 1);
                x = min(max(x, 0), a.W - 1);
            }
        }
        const Pt32 pt = locate32(a.in, (s * a.H + y) * a.W + x);
        const uint32_t edge = edge_dims32(a.in, pt);
        float v[CI];
#pragma unroll
        for (int f = 0; f < CI; ++f) {
            v[f] = 0.f;
            if (f < a.c0) {
                const int fix = edge ? edge_fix32(a.in, pt, a.tin.raw8[f], edge) : 0;
                v[f] = ldg(a.tin.fptr[f] + (pt.pe + fix));
            }
        }
        float4 *d4 = reinterpret_cast<float4 *>(dst + (size_t)i * CI);
#pragma unroll
        for (int c4 = 0; c4 < CI / 4; ++c4)
            d4[c4] = zero ? make_float4(0.f, 0.f, 0.f, 0.f)
                          : make_float4(v[4 * c4], v[4 * c4 + 1], v[4 * c4 + 2], v[4 * c4 + 3]);
    }
}

// One layer's launch constants, read from the kernel arguments with constant
// indices (a kernel-argument array indexed at run time would be copied to
// private memory first).
struct LayerRun {
    CnnFusedLayer Ly;
    int oh, ow, sw;        // output region; input region row length
    int rt, rl;            // output region origin relative to the tile
    int next_mode, last;
};

template <int l>
__device__ __forceinline__ LayerRun layer_run(const FusedArgs &a) {
    LayerRun r;
    r.Ly = a.L[l];
    r.oh = a.rh[l + 1];
    r.ow = a.rw[l + 1];
    r.sw = a.rw[l];
    r.rt = a.rt[l + 1];
    r.rl = a.rl[l + 1];
    r.last = l == a.n_layers - 1;
    r.next_mode = (l + 1 < kCnnFusedMaxLayers && !r.last) ? a.L[l + 1 < kCnnFusedMaxLayers ? l + 1 : l].mode
                                                          : HPACML_PADMODE_ZEROS;
    return r;
}

// One layer over its output region (the next layer's input region, or the tile).
template <int CIN4, int COUT4>
__device__ __forceinline__ void conv_pass(const FusedArgs &a, const LayerRun &r, const float *__restrict__ wts,
                                          const float *src, float *dst, int s, int y0, int x0) {
    constexpr int CI = 4 * CIN4, CO = 4 * COUT4;
    const CnnFusedLayer &Ly = r.Ly;
    const bool last = r.last;
    const int oh = r.oh, ow = r.ow, sw = r.sw;
    const int vy0 = y0 - r.rt, vx0 = x0 - r.rl;
    const int next_mode = r.next_mode;
    const float *wl = wts + Ly.woff;
    const float *bl = wts + Ly.boff;
    const int kh = Ly.kh, kw = Ly.kw;
    const int n = oh * ow;
    for (int i = threadIdx.x; i < n; i += kThreads) {
        int ry = i / ow, rx = i - ry * ow;
        const int vy = vy0 + ry, vx = vx0 + rx;
        const bool outside = vy < 0 || vy >= a.H || vx < 0 || vx >= a.W;
        bool zero = false;
        if (outside && !last && !a.circular) {
            if (next_mode == HPACML_PADMODE_REPLICATE) {
                ry = min(max(vy, 0), a.H - 1) - vy0;
                rx = min(max(vx, 0), a.W - 1) - vx0;
            } else {
                zero = true;
            }
        }
        float acc[CO];
#pragma unroll
        for (int co = 0; co < CO; ++co)
            acc[co] = bl[co];
        for (int ky = 0; ky < kh; ++ky) {
            const float *srow = src + (size_t)((ry + ky) * sw + rx) * CI;
            const float *wrow = wl + ky * kw * CI * CO;
            for (int kx = 0; kx < kw; ++kx) {
                const float4 *sp = reinterpret_cast<const float4 *>(srow + kx * CI);
                const float *wk = wrow + kx * CI * CO;
                float4 v[CIN4];
#pragma unroll
                for (int c4 = 0; c4 < CIN4; ++c4)
                    v[c4] = sp[c4];
#pragma unroll
                for (int c4 = 0; c4 < CIN4; ++c4) {
                    const float vv[4] = {v[c4].x, v[c4].y, v[c4].z, v[c4].w};
#pragma unroll
                    for (int ci = 0; ci < 4; ++ci)
#pragma unroll
                        for (int co = 0; co < CO; ++co)
                            acc[co] = fmaf(wk[(4 * c4 + ci) * CO + co], vv[ci], acc[co]);
                }
            }
        }
        if (Ly.act == HPACML_ACT_RELU) {
#pragma unroll
            for (int co = 0; co < CO; ++co)
                acc[co] = relu_arith(acc[co]);
        }
        if (last) {
            if (!outside) {
                const Pt32 pt = locate32(a.out, (s * a.H + vy) * a.W + vx);
                const uint32_t edge = edge_dims32(a.out, pt);
#pragma unroll
                for (int g = 0; g < CO; ++g)
                    if (g < a.cout_last) {
                        const int fix = edge ? edge_fix32(a.out, pt, a.tout.raw8[g], edge) : 0;
                        stg(const_cast<float *>(a.tout.fptr[g]) + (pt.pe + fix), acc[g]);
                    }
            }
        } else {
            float4 *d4 = reinterpret_cast<float4 *>(dst + (size_t)i * CO);
#pragma unroll
            for (int c4 = 0; c4 < COUT4; ++c4)
                d4[c4] = zero ? make_float4(0.f, 0.f, 0.f, 0.f)
                              : make_float4(acc[4 * c4], acc[4 * c4 + 1], acc[4 * c4 + 2], acc[4 * c4 + 3]);
        }
    }
}

template <int CIN4>
__device__ __forceinline__ void conv_dispatch_out(const FusedArgs &a, const LayerRun &r, const float *__restrict__ wts,
                                                  const float *src, float *dst, int s, int y0, int x0) {
    switch (r.Ly.cout4) {
    case 1: conv_pass<CIN4, 1>(a, r, wts, src, dst, s, y0, x0); break;
    case 2: conv_pass<CIN4, 2>(a, r, wts, src, dst, s, y0, x0); break;
    case 3: conv_pass<CIN4, 3>(a, r, wts, src, dst, s, y0, x0); break;
    default: conv_pass<CIN4, 4>(a, r, wts, src, dst, s, y0, x0); break;
    }
}

__global__ void __launch_bounds__(kThreads) cnn_fused_kernel(FusedArgs a, const float *__restrict__ wts) {
    extern __shared__ float4 lds4[];
    float *const buf0 = reinterpret_cast<float *>(lds4);
    float *const buf1 = buf0 + a.buf1;

    // blocks of one XCD (blockIdx % 8) take a contiguous range of tiles, so
    // neighbouring tiles share their halo rows in that XCD's L2
    const int32_t k0 = blockIdx.x;
    const int32_t xq = a.n_tiles / 8, xr = a.n_tiles % 8, xx = k0 % 8;
    const int32_t tile = xx * xq + (xx < xr ? xx : xr) + k0 / 8;
    const int32_t per_img = a.tiles_y * a.tiles_x;
    const int s = tile / per_img;
    const int rem = tile - s * per_img;
    const int ty_i = rem / a.tiles_x;
    const int y0 = ty_i * a.ty, x0 = (rem - ty_i * a.tiles_x) * kTX;

    switch (a.L[0].cin4) {
    case 1: gather_region<4>(a, s, y0, x0, buf0); break;
    case 2: gather_region<8>(a, s, y0, x0, buf0); break;
    case 3: gather_region<12>(a, s, y0, x0, buf0); break;
    default: gather_region<16>(a, s, y0, x0, buf0); break;
    }
    __syncthreads();
    for (int l = 0; l < a.n_layers; ++l) {
        LayerRun r;
        switch (l) {
        case 0: r = layer_run<0>(a); break;
        case 1: r = layer_run<1>(a); break;
        case 2: r = layer_run<2>(a); break;
        default: r = layer_run<3>(a); break;
        }
        const float *src = (l & 1) ? buf1 : buf0;
        float *dst = (l & 1) ? buf0 : buf1;
        switch (r.Ly.cin4) {
        case 1: conv_dispatch_out<1>(a, r, wts, src, dst, s, y0, x0); break;
        case 2: conv_dispatch_out<2>(a, r, wts, src, dst, s, y0, x0); break;
        case 3: conv_dispatch_out<3>(a, r, wts, src, dst, s, y0, x0); break;
        default: conv_dispatch_out<4>(a, r, wts, src, dst, s, y0, x0); break;
        }
        __syncthreads();
    }
}

// LDS floats of the two buffers for tiles of `ty` rows.
void fused_regions(const CnnFused &f, int ty, FusedArgs *a, size_t *floats0, size_t *floats1) {
    const int L = f.n_layers;
    a->rt[L] = a->rl[L] = 0;
    int rb = 0, rr = 0;
    a->rh[L] = ty;
    a->rw[L] = kTX;
    size_t b0 = 0, b1 = 0;
    for (int l = L - 1; l >= 0; --l) {
        const CnnFusedLayer &y = f.L[l];
        a->rt[l] = a->rt[l + 1] + y.top;
        a->rl[l] = a->rl[l + 1] + y.left;
        rb += y.kh - 1 - y.top;
        rr += y.kw - 1 - y.left;
        a->rh[l] = ty + a->rt[l] + rb;
        a->rw[l] = kTX + a->rl[l] + rr;
        const size_t fl = (size_t)a->rh[l] * a->rw[l] * 4 * y.cin4;
        if (l & 1)
            b1 = std::max(b1, fl);
        else
            b0 = std::max(b0, fl);
    }
    *floats0 = b0;
    *floats1 = b1;
}

constexpr size_t kLdsTwoBlocks = 64 * 1024;
constexpr size_t kLdsOneBlock = 160 * 1024;

// ------------------------------------------------------------------ layers
__global__ void __launch_bounds__(256) cnn_conv_kernel(CnnLayerDev L, const float *__restrict__ in,
                                                      float *__restrict__ out, int64_t total) {
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= total)
        return;
    const int co = (int)(idx % L.cout);
    const int64_t pix = idx / L.cout;
    const int ox = (int)(pix % L.w2);
    const int oy = (int)(pix / L.w2 % L.h2);
    const int64_t s = pix / ((int64_t)L.w2 * L.h2);
    const float *img = in + s * L.h * L.w * L.cin;
    const int y0 = oy * L.sh - (L.same ? (L.kh - 1) / 2 : 0);
    const int x0 = ox * L.sw - (L.same ? (L.kw - 1) / 2 : 0);
    float acc = L.b[co];
    for (int ky = 0; ky < L.kh; ++ky) {
        int y = y0 + ky;
        bool zy = false;
        if (y < 0 || y >= L.h) {
            if (L.mode == HPACML_PADMODE_CIRCULAR)
                y = wrap(y, L.h);
            else if (L.mode == HPACML_PADMODE_REPLICATE)
                y = min(max(y, 0), L.h - 1);
            else
                zy = true;
        }
        for (int kx = 0; kx < L.kw; ++kx) {
            int x = x0 + kx;
            bool z = zy;
            if (x < 0 || x >= L.w) {
                if (L.mode == HPACML_PADMODE_CIRCULAR)
                    x = wrap(x, L.w);
                else if (L.mode == HPACML_PADMODE_REPLICATE)
                    x = min(max(x, 0), L.w - 1);
                else
                    z = true;
            }
            if (z)
                continue;
            const float *px = img + ((int64_t)y * L.w + x) * L.cin;
            const float *wk = L.W + ((int64_t)co * L.cin * L.kh + ky) * L.kw + kx;
            for (int ci = 0; ci < L.cin; ++ci)
                acc = fmaf(wk[(int64_t)ci * L.kh * L.kw], px[ci], acc);
        }
    }
    out[idx] = L.act == HPACML_ACT_RELU ? (acc > 0.f ? acc : 0.f) : acc;
}

__global__ void __launch_bounds__(256) cnn_pool_kernel(CnnLayerDev L, const float *__restrict__ in,
                                                      float *__restrict__ out, int64_t total) {
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= total)
        return;
    const int c = (int)(idx % L.cout);
    const int64_t pix = idx / L.cout;
    const int ox = (int)(pix % L.w2);
    const int oy = (int)(pix / L.w2 % L.h2);
    const int64_t s = pix / ((int64_t)L.w2 * L.h2);
    const float *win = in + ((s * L.h + (int64_t)oy * L.sh) * L.w + (int64_t)ox * L.sw) * L.cin + c;
    // the largest window value; a NaN anywhere in the window wins
    float m = win[0];
    for (int ky = 0; ky < L.kh; ++ky)
        for (int kx = 0; kx < L.kw; ++kx) {
            const float v = win[((int64_t)ky * L.w + kx) * L.cin];
            if (!(m != m) && (v != v || v > m))
                m = v;
        }
    out[idx] = L.act == HPACML_ACT_RELU ? (m > 0.f ? m : 0.f) : m;
}

__global__ void __launch_bounds__(256) cnn_linear_kernel(CnnLayerDev L, const float *__restrict__ in,
                                                        float *__restrict__ out, int64_t total) {
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= total)
        return;
    const int o = (int)(idx % L.cout);
    const int64_t s = idx / L.cout;
    const int64_t n_in = (int64_t)L.h * L.w * L.cin;
    const float *x = in + s * n_in;
    const float *w = L.W + o * n_in;
    float acc = L.b[o];
    for (int64_t k = 0; k < n_in; ++k)
        acc = fmaf(w[k], x[k], acc);
    out[idx] = L.act == HPACML_ACT_RELU ? (acc > 0.f ? acc : 0.f) : acc;
}

__global__ void __launch_bounds__(256) scatter_record_kernel(DevMap m, const float *__restrict__ src) {
    const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= m.n_points)
        return;
    int64_t p[HPACML_MAX_RANK];
    sweep_point(m, b, p);
    const bool inside = interior(m, p);
    for (int g = 0; g < m.n_features; ++g)
        stg(const_cast<float *>(feature_ptr(m, p, inside, g)), src[b * m.n_features + g]);
}

}  // namespace

// ------------------------------------------------------------------ host
bool cnn_fused_supported(const CnnPlan &p) {
    if (p.n_layers > kCnnFusedMaxLayers)
        return false;
    int circ = 0;
    for (int l = 0; l < p.n_layers; ++l) {
        const hpacml_layer &y = p.layers[l];
        if (y.kind != HPACML_LAYER_CONV2D || y.padding != HPACML_PAD_SAME || y.kernel[0] > 16 || y.kernel[1] > 16)
            return false;
        if (p.shape[l].c > kCnnFusedMaxC || p.shape[l + 1].c > kCnnFusedMaxC)
            return false;
        circ += y.pad_mode == HPACML_PADMODE_CIRCULAR;
    }
    return circ == 0 || circ == p.n_layers;
}

void cnn_fused_pack(const CnnPlan &p, const float *const *W, const float *const *b, std::vector<float> &buf,
                    CnnFused *out) {
    CnnFused f{};
    f.n_layers = p.n_layers;
    f.c0 = p.in_channels;
    f.cout_last = p.shape[p.n_layers].c;
    f.circular = p.layers[0].pad_mode == HPACML_PADMODE_CIRCULAR;
    buf.clear();
    for (int l = 0; l < p.n_layers; ++l) {
        const hpacml_layer &y = p.layers[l];
        CnnFusedLayer &d = f.L[l];
        const int cin = p.shape[l].c, cout = p.shape[l + 1].c;
        d.cin4 = (cin + 3) / 4;
        d.cout4 = (cout + 3) / 4;
        d.kh = y.kernel[0];
        d.kw = y.kernel[1];
        d.top = (d.kh - 1) / 2;
        d.left = (d.kw - 1) / 2;
        d.act = y.act;
        d.mode = y.pad_mode;
        const int CI = 4 * d.cin4, CO = 4 * d.cout4;
        // [ky][kx][ci][co], zero in the padded channels
        d.woff = (int32_t)buf.size();
        buf.resize(buf.size() + (size_t)d.kh * d.kw * CI * CO, 0.f);
        for (int co = 0; co < cout; ++co)
            for (int ci = 0; ci < cin; ++ci)
                for (int ky = 0; ky < d.kh; ++ky)
                    for (int kx = 0; kx < d.kw; ++kx)
                        buf[d.woff + (((size_t)ky * d.kw + kx) * CI + ci) * CO + co] =
                            W[l][(((size_t)co * cin + ci) * d.kh + ky) * d.kw + kx];
        d.boff = (int32_t)buf.size();
        buf.resize(buf.size() + CO, 0.f);
        for (int co = 0; co < cout; ++co)
            buf[d.boff + co] = b[l][co];
    }
    *out = f;
}

int cnn_fused_tile_rows(const CnnFused &f, int32_t H) {
    // the largest tile of at most max(H, 1) rows (rounded up to a power of
    // two) whose buffers leave room for two blocks per CU, else for one
    int one = 0;
    for (int ty : {32, 16, 8, 4, 2, 1}) {
        if (ty > 1 && ty / 2 >= H)
            continue;
        FusedArgs a{};
        size_t f0, f1;
        fused_regions(f, ty, &a, &f0, &f1);
        const size_t bytes = (f0 + f1) * sizeof(float);
        if (bytes <= kLdsTwoBlocks)
            return ty;
        if (!one && bytes <= kLdsOneBlock)
            one = ty;
    }
    return one;
}

hipError_t launch_cnn_fused(const Map32 &in, const Map32 &out, const FeatTable32 &tin, const FeatTable32 &tout,
                            const CnnFused &f, int32_t S, int32_t H, int32_t W, hipStream_t stream) {
    const int ty = cnn_fused_tile_rows(f, H);
    if (ty == 0)
        return hipErrorInvalidValue;
    FusedArgs a{};
    a.in = in;
    a.out = out;
    a.tin = tin;
    a.tout = tout;
    a.S = S;
    a.H = H;
    a.W = W;
    a.n_layers = f.n_layers;
    a.ty = ty;
    a.tiles_y = (H + ty - 1) / ty;
    a.tiles_x = (W + kTX - 1) / kTX;
    const int64_t n_tiles = (int64_t)S * a.tiles_y * a.tiles_x;
    if (n_tiles == 0)
        return hipSuccess;
    if (n_tiles > INT32_MAX)
        return hipErrorInvalidValue;
    a.n_tiles = (int32_t)n_tiles;
    a.c0 = f.c0;
    a.cout_last = f.cout_last;
    a.circular = f.circular;
    for (int l = 0; l < f.n_layers; ++l)
        a.L[l] = f.L[l];
    size_t f0, f1;
    fused_regions(f, ty, &a, &f0, &f1);
    a.buf1 = (int32_t)f0;
    const size_t lds = (f0 + f1) * sizeof(float);
    hipError_t e = hipFuncSetAttribute((const void *)cnn_fused_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)lds);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(cnn_fused_kernel, dim3((unsigned)n_tiles), dim3(kThreads), lds, stream, a, f.wts);
    return hipGetLastError();
}

hipError_t launch_cnn_layer(const CnnLayerDev &L, const float *in, float *out, int64_t S, hipStream_t stream) {
    const int64_t total = S * (int64_t)L.h2 * L.w2 * L.cout;
    if (total == 0)
        return hipSuccess;
    const int64_t blocks = (total + 255) / 256;
    if (blocks > INT32_MAX)
        return hipErrorInvalidValue;
    switch (L.kind) {
    case HPACML_LAYER_CONV2D:
        hipLaunchKernelGGL(cnn_conv_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, L, in, out, total);
        break;
    case HPACML_LAYER_MAXPOOL2D:
        hipLaunchKernelGGL(cnn_pool_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, L, in, out, total);
        break;
    default:
        hipLaunchKernelGGL(cnn_linear_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, L, in, out, total);
        break;
    }
    return hipGetLastError();
}

hipError_t launch_scatter_record(const DevMap &m, const float *src, hipStream_t stream) {
    if (m.n_points == 0)
        return hipSuccess;
    const int64_t blocks = (m.n_points + 255) / 256;
    if (blocks > INT32_MAX)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(scatter_record_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, m, src);
    return hipGetLastError();
}

}  // namespace hpacml
