// Convolutional surrogates on the composed tensor seen as images (Table IV
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
// layer's input region — and finally writes the last layer's tile through the
// `from` map (a phase of its own, so the layer loops carry none of the output
// map's state in registers).  One thread computes one pixel's output
// channels per pass: 16-byte LDS reads of its window, weights as wave-uniform
// scalar loads (one FMA per weight per lane), no bank conflicts for 4-channel
// rows.  Outside the image, a layer's input follows its padding mode:
// circular stacks wrap at the gather and then compute the halo as is (on a
// torus the halo's values equal the wrapped ones); zeros writes 0; replicate
// computes the pixel at the clamped position (inside the region, since the
// region always contains the image edge it crosses).
//
// Layer-by-layer path (everything else, and in-place regions): kernels over
// [S][h][w][c] tensors in a workspace -- convolutions (a max-pool with
// non-overlapping windows folded into the convolution before it), pools,
// fully connected layers (split K when the tiles alone are too few), and the
// fully connected layers closing a stack together with the scatter; else a
// scatter of the last tensor.
#include "cnn.hpp"

namespace hpacml {

namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int kTX = 64;   // tile columns
constexpr int kPix = 1;   // pixels per thread per pass

// ------------------------------------------------------------------ fused
struct FusedArgs {
    Map32 in, out;
    const FeatTable32 *tin, *tout;   // device; the used entries are staged in LDS
    int32_t S, H, W, n_layers;
    int32_t ty, tiles_x, tiles_y, n_tiles;
    int32_t c0, cout_last, circular, buf1;   // buf1: float offset of the second LDS buffer
    int32_t co_last_pad;                     // the last layer's channels, padded to 4
    // region of layer l's input (l = n_layers: the tile itself), relative to
    // the tile origin: rows [-rt, ty + rb), columns [-rl, 64 + rr)
    int32_t rt[kCnnFusedMaxLayers + 1], rl[kCnnFusedMaxLayers + 1];
    int32_t rh[kCnnFusedMaxLayers + 1], rw[kCnnFusedMaxLayers + 1];
    uint32_t rw_magic[kCnnFusedMaxLayers + 1];   // i / rw == (i * rw_magic) >> 24 for i < 2^16
    CnnFusedLayer L[kCnnFusedMaxLayers];
};

// Feature tables of the two maps in LDS (the first 16 entries): read with a
// wave-uniform index, so every lane gets the same pointer, without holding
// 16 pointers per map in scalar registers for the whole kernel.
struct TabLds {
    const float *in[kCnnFusedMaxC];
    float *out[kCnnFusedMaxC];
    uint32_t in_raw8[kCnnFusedMaxC], out_raw8[kCnnFusedMaxC];
};

__device__ __forceinline__ int div_region(int i, uint32_t magic) { return (int)(((uint32_t)i * magic) >> 24); }

__device__ __forceinline__ int wrap(int v, int n) {
    int r = v % n;
    return r < 0 ? r + n : r;
}

// Layer 0's input region from the `to` map: pixel (y, x) of image s is
// composed point (s * H + y) * W + x; channel f is its feature f.
template <int CI>
__device__ __forceinline__ void gather_region(const FusedArgs &a, const TabLds &tab, int s, int y0, int x0,
                                              float *dst) {
    const int rh = a.rh[0], rw = a.rw[0], n = rh * rw;
    const int mode = a.L[0].mode;
    const int vy0 = y0 - a.rt[0], vx0 = x0 - a.rl[0];
    for (int i = threadIdx.x; i < n; i += kThreads) {
        const int ry = div_region(i, a.rw_magic[0]), rx = i - ry * rw;
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
                const int fix = edge ? edge_fix32(a.in, pt, tab.in_raw8[f], edge) : 0;
                v[f] = ldg(tab.in[f] + (pt.pe + fix));
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
    uint32_t ow_magic;
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
    r.ow_magic = a.rw_magic[l + 1];
    r.rt = a.rt[l + 1];
    r.rl = a.rl[l + 1];
    r.last = l == a.n_layers - 1;
    r.next_mode = (l + 1 < kCnnFusedMaxLayers && !r.last) ? a.L[l + 1 < kCnnFusedMaxLayers ? l + 1 : l].mode
                                                          : HPACML_PADMODE_ZEROS;
    return r;
}

// One layer over its output region (the next layer's input region, or the
// tile for the last layer) into LDS.  Each thread takes kPix pixels per pass
// (i, i + kThreads, ...): a weight loaded once feeds kPix FMAs.  Pixels
// outside the image get what the next layer's padding reads there (the last
// layer's are never stored).
template <int CIN4, int COUT4>
__device__ __forceinline__ void conv_pass(const FusedArgs &a, const TabLds &tab, const LayerRun &r,
                                          const float *__restrict__ wts, const float *src, float *dst, int s, int y0,
                                          int x0) {
    constexpr int CI = 4 * CIN4, CO = 4 * COUT4;
    const CnnFusedLayer &Ly = r.Ly;
    const int oh = r.oh, ow = r.ow, sw = r.sw;
    const int vy0 = y0 - r.rt, vx0 = x0 - r.rl;
    const int next_mode = r.next_mode;
    const float *wl = wts + Ly.woff;
    const float *bl = wts + Ly.boff;
    const int kh = Ly.kh, kw = Ly.kw;
    const int n = oh * ow;
    for (int base = 0; base < n; base += kThreads * kPix) {
        int off[kPix];          // LDS float offset of each pixel's window origin
        bool valid[kPix], zero[kPix];
#pragma unroll
        for (int j = 0; j < kPix; ++j) {
            const int i = base + j * kThreads + (int)threadIdx.x;
            valid[j] = i < n;
            const int ic = valid[j] ? i : n - 1;
            int ry = div_region(ic, r.ow_magic), rx = ic - ry * ow;
            const int vy = vy0 + ry, vx = vx0 + rx;
            const bool outside = vy < 0 || vy >= a.H || vx < 0 || vx >= a.W;
            zero[j] = false;
            if (outside && !a.circular) {
                if (next_mode == HPACML_PADMODE_REPLICATE) {
                    ry = min(max(vy, 0), a.H - 1) - vy0;
                    rx = min(max(vx, 0), a.W - 1) - vx0;
                } else {
                    zero[j] = true;
                }
            }
            off[j] = (ry * sw + rx) * CI;
        }
        // output channels in groups of 4, one group at a time: a step (kx,
        // 4 input channels) then holds 16 weights in scalar registers, which
        // leaves the registers the pass's other uniform values need (larger
        // weight sets spilled them); the window is re-read from LDS per group
        const int nq = kw * CIN4;
#pragma unroll 1
        for (int og = 0; og < COUT4; ++og) {
            const float *wg = wl + og * kh * nq * 16;
            float acc[kPix][4];
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const float bv = bl[4 * og + c];
#pragma unroll
                for (int j = 0; j < kPix; ++j)
                    acc[j][c] = bv;
            }
            for (int ky = 0; ky < kh; ++ky) {
                const float *wrow = wg + ky * nq * 16;
                const int rowoff = ky * sw * CI;
                for (int q = 0; q < nq; ++q) {
                    const float *wk = wrow + q * 16;
                    float4 v[kPix];
#pragma unroll
                    for (int j = 0; j < kPix; ++j)
                        v[j] = *reinterpret_cast<const float4 *>(src + off[j] + rowoff + 4 * q);
#pragma unroll
                    for (int ci = 0; ci < 4; ++ci)
#pragma unroll
                        for (int c = 0; c < 4; ++c) {
                            const float wv = wk[ci * 4 + c];
#pragma unroll
                            for (int j = 0; j < kPix; ++j) {
                                const float x = ci == 0 ? v[j].x : ci == 1 ? v[j].y : ci == 2 ? v[j].z : v[j].w;
                                acc[j][c] = fmaf(wv, x, acc[j][c]);
                            }
                        }
                }
            }
#pragma unroll
            for (int j = 0; j < kPix; ++j) {
                if (Ly.act == HPACML_ACT_RELU) {
#pragma unroll
                    for (int c = 0; c < 4; ++c)
                        acc[j][c] = relu_arith(acc[j][c]);
                }
                if (!valid[j])
                    continue;
                const int i = base + j * kThreads + (int)threadIdx.x;
                reinterpret_cast<float4 *>(dst + (size_t)i * CO)[og] =
                    zero[j] ? make_float4(0.f, 0.f, 0.f, 0.f) : make_float4(acc[j][0], acc[j][1], acc[j][2], acc[j][3]);
            }
        }
    }
}

// The last layer's tile (LDS, [pixel][4 * cout4]) through the `from` map:
// pixel (y, x) of image s is point (s * H + y) * W + x, channel g its feature g.
__device__ __forceinline__ void scatter_tile(const FusedArgs &a, const TabLds &tab, const float *src, int s, int y0,
                                             int x0) {
    const int CO = a.co_last_pad;
    const int n = a.ty * kTX;
    for (int i = threadIdx.x; i < n; i += kThreads) {
        const int ry = i / kTX, rx = i % kTX;
        const int y = y0 + ry, x = x0 + rx;
        if (y >= a.H || x >= a.W)
            continue;
        const Pt32 pt = locate32(a.out, (s * a.H + y) * a.W + x);
        const uint32_t edge = edge_dims32(a.out, pt);
        const float *v = src + (size_t)i * CO;
        for (int g = 0; g < a.cout_last; ++g) {
            const int fix = edge ? edge_fix32(a.out, pt, tab.out_raw8[g], edge) : 0;
            stg(tab.out[g] + (pt.pe + fix), v[g]);
        }
    }
}

template <int CIN4>
__device__ __forceinline__ void conv_dispatch_out(const FusedArgs &a, const TabLds &tab, const LayerRun &r,
                                                  const float *__restrict__ wts, const float *src, float *dst, int s,
                                                  int y0, int x0) {
    switch (r.Ly.cout4) {
    case 1: conv_pass<CIN4, 1>(a, tab, r, wts, src, dst, s, y0, x0); break;
    case 2: conv_pass<CIN4, 2>(a, tab, r, wts, src, dst, s, y0, x0); break;
    case 3: conv_pass<CIN4, 3>(a, tab, r, wts, src, dst, s, y0, x0); break;
    default: conv_pass<CIN4, 4>(a, tab, r, wts, src, dst, s, y0, x0); break;
    }
}

__global__ void __launch_bounds__(kThreads) cnn_fused_kernel(FusedArgs a, const float *__restrict__ wts) {
    extern __shared__ float4 lds4[];
    float *const buf0 = reinterpret_cast<float *>(lds4);
    float *const buf1 = buf0 + a.buf1;
    __shared__ TabLds tab;
    if (threadIdx.x < kCnnFusedMaxC) {
        const int f = threadIdx.x;
        tab.in[f] = a.tin->fptr[f];
        tab.in_raw8[f] = a.tin->raw8[f];
        tab.out[f] = const_cast<float *>(a.tout->fptr[f]);
        tab.out_raw8[f] = a.tout->raw8[f];
    }
    __syncthreads();

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
    case 1: gather_region<4>(a, tab, s, y0, x0, buf0); break;
    case 2: gather_region<8>(a, tab, s, y0, x0, buf0); break;
    case 3: gather_region<12>(a, tab, s, y0, x0, buf0); break;
    default: gather_region<16>(a, tab, s, y0, x0, buf0); break;
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
        case 1: conv_dispatch_out<1>(a, tab, r, wts, src, dst, s, y0, x0); break;
        case 2: conv_dispatch_out<2>(a, tab, r, wts, src, dst, s, y0, x0); break;
        case 3: conv_dispatch_out<3>(a, tab, r, wts, src, dst, s, y0, x0); break;
        default: conv_dispatch_out<4>(a, tab, r, wts, src, dst, s, y0, x0); break;
        }
        __syncthreads();
    }
    scatter_tile(a, tab, (a.n_layers & 1) ? buf1 : buf0, s, y0, x0);
}

// LDS floats of the two buffers for tiles of `ty` rows.
void fused_regions(const CnnFused &f, int ty, FusedArgs *a, size_t *floats0, size_t *floats1) {
    const int L = f.n_layers;
    a->rt[L] = a->rl[L] = 0;
    int rb = 0, rr = 0;
    a->rh[L] = ty;
    a->rw[L] = kTX;
    size_t b0 = 0, b1 = 0;
    // the last layer's output tile
    ((L & 1) ? b1 : b0) = (size_t)ty * kTX * 4 * f.L[L - 1].cout4;
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

// tile buffers of at most 40 KB leave room for four blocks (16 waves) per CU:
// measured faster than 64 KB tiles with two blocks, the recomputed halo
// notwithstanding
constexpr size_t kLdsShared = 40 * 1024;
constexpr size_t kLdsOneBlock = 160 * 1024;

// ------------------------------------------------------------------ layers
// One thread per output pixel and group of kConvG output channels
// (blockIdx.y).  Weights packed [group][ky][kx][ci][kConvG], zero past cout:
// in the channels-last image the taps of one window row are one contiguous
// run of kw * cin floats, and the kConvG weights of a tap are one
// wave-uniform 32-byte scalar load, so every input value read feeds kConvG
// FMAs.  Taps go in chunks of kTapChunk whose input loads are all issued
// before the first FMA.  A pixel whose window leaves the image (SAME
// padding at the border) resolves each tap through the padding mode.
//
// With POOL, a max-pool whose windows do not overlap follows in the same
// kernel, so the convolution's output never goes to memory: a group of
// 2^qshift adjacent lanes holds one pooled pixel, lane q computing window
// position q (lanes past the window repeat position 0), and the group's
// maximum comes from xor shuffles.  Each pairwise step keeps the lower
// lane's value unless the other is larger or a NaN, and a NaN once taken
// stays: the window's first NaN, else its first maximum, as in the pool
// kernel.
constexpr int kTapChunk = 16;

// Convolution outputs (bias, taps, activation) of output pixel (oy, ox).
__device__ __forceinline__ void conv_pixel(const CnnLayerDev &L, const float *img, const float *__restrict__ wg,
                                           int oy, int ox, int ng, float (&acc)[kConvG]) {
    const int y0 = oy * L.sh - (L.same ? (L.kh - 1) / 2 : 0);
    const int x0 = ox * L.sw - (L.same ? (L.kw - 1) / 2 : 0);
    const int taps = L.kh * L.kw * L.cin;
#pragma unroll
    for (int g = 0; g < kConvG; ++g)
        acc[g] = g < ng ? L.b[blockIdx.y * kConvG + g] : 0.f;
    if (y0 >= 0 && x0 >= 0 && y0 + L.kh <= L.h && x0 + L.kw <= L.w) {
        const float *base = img + ((int64_t)y0 * L.w + x0) * L.cin;
        const int run = L.kw * L.cin;                 // floats of one window row
        const int64_t rs = (int64_t)L.w * L.cin;      // image row stride
        int ky = 0, r = 0;
        if (run % 4 == 0 && rs % 4 == 0 && ((uintptr_t)base & 15) == 0) {
            // window rows of whole, aligned float4s: 16-byte loads
            for (int t0 = 0; t0 < taps; t0 += kTapChunk) {
                float4 v[kTapChunk / 4];
#pragma unroll
                for (int j = 0; j < kTapChunk / 4; ++j) {
                    v[j] = t0 + 4 * j < taps ? *reinterpret_cast<const float4 *>(base + ky * rs + r)
                                             : make_float4(0.f, 0.f, 0.f, 0.f);
                    r += 4;
                    if (r == run) {
                        r = 0;
                        ++ky;
                    }
                }
#pragma unroll
                for (int j = 0; j < kTapChunk / 4; ++j)
                    if (t0 + 4 * j < taps) {
                        const float *w = wg + (int64_t)(t0 + 4 * j) * kConvG;
                        const float e[4] = {v[j].x, v[j].y, v[j].z, v[j].w};
#pragma unroll
                        for (int i = 0; i < 4; ++i)
#pragma unroll
                            for (int g = 0; g < kConvG; ++g)
                                acc[g] = fmaf(w[i * kConvG + g], e[i], acc[g]);
                    }
            }
        } else
        for (int t0 = 0; t0 < taps; t0 += kTapChunk) {
            float v[kTapChunk];
#pragma unroll
            for (int j = 0; j < kTapChunk; ++j) {
                v[j] = t0 + j < taps ? base[ky * rs + r] : 0.f;
                if (++r == run) {
                    r = 0;
                    ++ky;
                }
            }
#pragma unroll
            for (int j = 0; j < kTapChunk; ++j)
                if (t0 + j < taps) {
                    const float *w = wg + (int64_t)(t0 + j) * kConvG;
#pragma unroll
                    for (int g = 0; g < kConvG; ++g)
                        acc[g] = fmaf(w[g], v[j], acc[g]);
                }
        }
    } else {
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
                const float *wk = wg + (int64_t)(ky * L.kw + kx) * L.cin * kConvG;
                for (int ci = 0; ci < L.cin; ++ci) {
                    const float v = px[ci];
#pragma unroll
                    for (int g = 0; g < kConvG; ++g)
                        acc[g] = fmaf(wk[ci * kConvG + g], v, acc[g]);
                }
            }
        }
    }
#pragma unroll
    for (int g = 0; g < kConvG; ++g)
        acc[g] = L.act == HPACML_ACT_RELU ? (acc[g] > 0.f ? acc[g] : 0.f) : acc[g];
}

__device__ __forceinline__ uint32_t fdiv(uint32_t i, uint32_t magic, uint32_t shift) {
    return (uint32_t)(((uint64_t)i * magic) >> shift);
}

template <bool POOL>
__global__ void __launch_bounds__(256) cnn_conv_kernel(CnnLayerDev L, CnnLayerDev P, int qshift,
                                                      const float *__restrict__ in, float *__restrict__ out,
                                                      int64_t n_pix) {
    const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t pix = POOL ? tid >> qshift : tid;
    if (!POOL && pix >= n_pix)
        return;
    // (pooled: every lane of a group takes part in the shuffles)
    const int64_t pc = pix < n_pix ? pix : n_pix - 1;
    const int co0 = blockIdx.y * kConvG;
    const int ng = min(kConvG, L.cout - co0);
    const CnnLayerDev &G = POOL ? P : L;   // the grid of output pixels
    int ox, oy;
    int64_t s;
    if (n_pix <= INT32_MAX) {
        // 32-bit divisions by multiply-shift (a 64-bit division is a long
        // instruction sequence, and this kernel is VALU-bound)
        const uint32_t q1 = fdiv((uint32_t)pc, G.w2_magic, G.w2_shift);
        const uint32_t q2 = fdiv(q1, G.h2_magic, G.h2_shift);
        ox = (int)((uint32_t)pc - q1 * (uint32_t)G.w2);
        oy = (int)(q1 - q2 * (uint32_t)G.h2);
        s = q2;
    } else {
        ox = (int)(pc % G.w2);
        oy = (int)(pc / G.w2 % G.h2);
        s = pc / ((int64_t)G.w2 * G.h2);
    }
    const int q = POOL ? (int)(tid & ((1 << qshift) - 1)) : 0;
    if (POOL) {
        // window position qq < 16 of a window kw <= 16 wide: (qq + 1/2) / kw
        // lies at least 1/32 from an integer, so the approximate reciprocal
        // gives the exact quotient
        const int qq = q < P.kh * P.kw ? q : 0;
        const int qy = (int)(((float)qq + 0.5f) * __builtin_amdgcn_rcpf((float)P.kw));
        oy = oy * P.sh + qy;
        ox = ox * P.sw + (qq - qy * P.kw);
    }
    const float *img = in + s * L.h * L.w * L.cin;
    const float *__restrict__ wg = L.W + (int64_t)blockIdx.y * L.kh * L.kw * L.cin * kConvG;
    float acc[kConvG];
    conv_pixel(L, img, wg, oy, ox, ng, acc);
    if (POOL) {
        for (int d = 1; d < (1 << qshift); d <<= 1) {
            const bool lower = (q & d) == 0;
#pragma unroll
            for (int g = 0; g < kConvG; ++g) {
                const float o = __shfl_xor(acc[g], d);
                const float a = lower ? acc[g] : o, b = lower ? o : acc[g];
                acc[g] = (!(a != a) && (b != b || b > a)) ? b : a;
            }
        }
#pragma unroll
        for (int g = 0; g < kConvG; ++g)
            acc[g] = P.act == HPACML_ACT_RELU ? (acc[g] > 0.f ? acc[g] : 0.f) : acc[g];
        if (q != 0 || pix >= n_pix)
            return;
    }
    float *o = out + pix * L.cout + co0;
    if (ng == kConvG && ((uintptr_t)o & 15) == 0) {
        *reinterpret_cast<float4 *>(o) = make_float4(acc[0], acc[1], acc[2], acc[3]);
        *reinterpret_cast<float4 *>(o + 4) = make_float4(acc[4], acc[5], acc[6], acc[7]);
    } else {
        for (int g = 0; g < ng; ++g)
            o[g] = acc[g];
    }
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

// Fully connected layer over S images: out[S][O] = in[S][K] W^T + b.  A block
// owns a T x T output tile (T = 64: 4 x 4 outputs per thread; T = 16 for
// layers of at most 16 outputs, one output per thread), K in chunks staged in
// LDS k-major, coalesced loads along k.
// Split-K: block z of gridDim.z sums k in [z Kc, (z+1) Kc) and, when
// gridDim.z > 1, writes its raw partial sums to part[z][S][O] (a reduce kernel
// adds them in z order, then bias and activation).
template <int T>
__global__ void __launch_bounds__(256) cnn_linear_kernel(CnnLayerDev L, const float *__restrict__ in,
                                                        float *__restrict__ out, int64_t S, int64_t Kc,
                                                        float *__restrict__ part) {
    constexpr int R = T / 16;                 // outputs per thread per dimension
    constexpr int KC = 256 * 4 / T;           // k per chunk: each thread loads 4 values per operand
    __shared__ float xs[KC][T + 4];
    __shared__ float ws[KC][T + 4];
    const int t = threadIdx.x;
    const int64_t s0 = (int64_t)blockIdx.x * T;
    const int o0 = blockIdx.y * T;
    const int O = L.cout;
    const int64_t K = (int64_t)L.h * L.w * L.cin;
    const int ti = t / 16, tj = t % 16;
    const int64_t kb = (int64_t)blockIdx.z * Kc;
    const int64_t ke = kb + Kc < K ? kb + Kc : K;
    float acc[R][R] = {};
    // T rows x KC columns of each operand per chunk: thread t loads column
    // t % KC of rows t / KC + (256 / KC) m, into registers one chunk ahead
    const int c = t % KC;
    float xr[4], wr[4];
    auto fetch = [&](int64_t k0) {
        const int64_t k = k0 + c;
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            const int r = t / KC + (256 / KC) * m;
            const int64_t sr = s0 + r;
            const int o = o0 + r;
            xr[m] = (sr < S && k < ke) ? in[sr * K + k] : 0.f;
            wr[m] = (o < O && k < ke) ? L.W[(int64_t)o * K + k] : 0.f;
        }
    };
    if (kb < ke)
        fetch(kb);
    for (int64_t k0 = kb; k0 < ke; k0 += KC) {
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            const int r = t / KC + (256 / KC) * m;
            xs[c][r] = xr[m];
            ws[c][r] = wr[m];
        }
        __syncthreads();
        if (k0 + KC < ke)
            fetch(k0 + KC);
#pragma unroll 8
        for (int kk = 0; kk < KC; ++kk) {
            float a[R], b[R];
#pragma unroll
            for (int i = 0; i < R; ++i) {
                a[i] = xs[kk][R * ti + i];
                b[i] = ws[kk][R * tj + i];
            }
#pragma unroll
            for (int i = 0; i < R; ++i)
#pragma unroll
                for (int j = 0; j < R; ++j)
                    acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < R; ++i) {
        const int64_t sr = s0 + R * ti + i;
        if (sr >= S)
            continue;
#pragma unroll
        for (int j = 0; j < R; ++j) {
            const int o = o0 + R * tj + j;
            if (o < O) {
                if (gridDim.z > 1) {
                    part[((int64_t)blockIdx.z * S + sr) * O + o] = acc[i][j];
                } else {
                    const float v = acc[i][j] + L.b[o];
                    out[sr * O + o] = L.act == HPACML_ACT_RELU ? (v > 0.f ? v : 0.f) : v;
                }
            }
        }
    }
}

// The products of a fully connected layer with more than 16 outputs whose K
// is split over blocks, on fp32 MFMA (v_mfma_f32_32x32x2f32): the transposed
// product C[o][s] = sum_k W[o][k] in[s][k], weights as the A operand (32
// outputs x 2 k per m-block), images as B (32 images x 2 k).  A block of 4
// waves owns 128 images (32 per wave) x 64 outputs (2 m-blocks) and one K
// range; K goes in chunks of kMfK staged in LDS (rows padded to kMfK + 1
// floats: lane l reads row l % 32 at column k + l / 32, conflict-free),
// loaded one chunk ahead in registers.  Lane l ends up holding image l % 32
// and, in register r of m-block mb, output 32 mb + 8 (r / 4) + 4 (l / 32) +
// r % 4: four consecutive outputs per group of registers, stored as one
// 16-byte write of the raw partial sums part[z][s][o].
constexpr int kMfS = 128, kMfO = 64, kMfK = 32;

__global__ void __launch_bounds__(256) cnn_linear_mfma_kernel(CnnLayerDev L, const float *__restrict__ in, int64_t S,
                                                             int64_t Kc, float *__restrict__ part) {
    __shared__ float xs[kMfS][kMfK + 1];
    __shared__ float ws[kMfO][kMfK + 1];
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    const int64_t s0 = (int64_t)blockIdx.x * kMfS;
    const int o0 = blockIdx.y * kMfO;
    const int O = L.cout;
    const int64_t K = (int64_t)L.h * L.w * L.cin;
    const int64_t kb = (int64_t)blockIdx.z * Kc;
    const int64_t ke = kb + Kc < K ? kb + Kc : K;
    // chunk loads: thread t takes column t % 32 of rows t / 32 + 8 m
    const int c = t % kMfK, r0 = t / kMfK;
    float xr[kMfS / 8], wr[kMfO / 8];
    auto fetch = [&](int64_t k0) {
        const int64_t k = k0 + c;
        const bool kin = k < ke;
#pragma unroll
        for (int m = 0; m < kMfS / 8; ++m) {
            const int64_t sr = s0 + r0 + 8 * m;
            xr[m] = (kin && sr < S) ? in[sr * K + k] : 0.f;
        }
#pragma unroll
        for (int m = 0; m < kMfO / 8; ++m) {
            const int o = o0 + r0 + 8 * m;
            wr[m] = (kin && o < O) ? L.W[(int64_t)o * K + k] : 0.f;
        }
    };
    floatx16 acc[2];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r)
            acc[mb][r] = 0.f;
    if (kb < ke)
        fetch(kb);
    const int col = lane & 31, kh = lane >> 5;
    for (int64_t k0 = kb; k0 < ke; k0 += kMfK) {
#pragma unroll
        for (int m = 0; m < kMfS / 8; ++m)
            xs[r0 + 8 * m][c] = xr[m];
#pragma unroll
        for (int m = 0; m < kMfO / 8; ++m)
            ws[r0 + 8 * m][c] = wr[m];
        __syncthreads();
        if (k0 + kMfK < ke)
            fetch(k0 + kMfK);
#pragma unroll
        for (int kk = 0; kk < kMfK; kk += 2) {
            const float b = xs[32 * w + col][kk + kh];
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
                acc[mb] = __builtin_amdgcn_mfma_f32_32x32x2f32(ws[32 * mb + col][kk + kh], b, acc[mb], 0, 0, 0);
        }
        __syncthreads();
    }
    const int64_t s = s0 + 32 * w + col;
    if (s >= S)
        return;
    float *dst = part + ((int64_t)blockIdx.z * S + s) * O;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int o = o0 + 32 * mb + 8 * q + 4 * kh;
            if (o + 3 < O && ((uintptr_t)(dst + o) & 15) == 0) {
                *reinterpret_cast<float4 *>(dst + o) =
                    make_float4(acc[mb][4 * q], acc[mb][4 * q + 1], acc[mb][4 * q + 2], acc[mb][4 * q + 3]);
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (o + i < O)
                        dst[o + i] = acc[mb][4 * q + i];
            }
        }
}

__global__ void __launch_bounds__(256) cnn_linear_reduce_kernel(CnnLayerDev L, const float *__restrict__ part,
                                                               float *__restrict__ out, int64_t S, int splits) {
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t n = S * L.cout;
    if (idx >= n)
        return;
    float v = 0.f;
#pragma unroll 8
    for (int z = 0; z < splits; ++z)
        v += part[z * n + idx];
    v += L.b[idx % L.cout];
    out[idx] = L.act == HPACML_ACT_RELU ? (v > 0.f ? v : 0.f) : v;
}

// The fully connected layers that end a stack, once the first of them has
// run its products: a block of 256 threads takes 256 / width images (width =
// the widest of these layers), adds the first layer's partial sums in block
// order with bias and activation (or reads its finished outputs), runs the
// remaining small layers on vectors in LDS (thread (image, o) computes
// output o in k order, then adds the bias), and scatters the last layer's
// outputs through the `from` map (one point per image).
__global__ void __launch_bounds__(256) cnn_tail_kernel(CnnTail T, const float *__restrict__ src, DevMap m,
                                                      int64_t S) {
    __shared__ float buf[2][256];
    const int ws = T.width;
    const int sb = threadIdx.x / ws, o = threadIdx.x % ws;
    const int64_t s = (int64_t)blockIdx.x * (256 / ws) + sb;
    const bool live = sb < 256 / ws && s < S;
    {
        const CnnLayerDev &L = T.first;
        if (live && o < L.cout) {
            float v;
            if (T.splits) {
                const int64_t n = S * L.cout, idx = s * L.cout + o;
                // every partial in flight before the first add; the sum in block order
                float pv[kLinSplit];
#pragma unroll
                for (int z = 0; z < kLinSplit; ++z)
                    pv[z] = z < T.splits ? src[z * n + idx] : 0.f;
                v = 0.f;
#pragma unroll
                for (int z = 0; z < kLinSplit; ++z)
                    if (z < T.splits)
                        v += pv[z];
                v += L.b[o];
                v = L.act == HPACML_ACT_RELU ? (v > 0.f ? v : 0.f) : v;
            } else {
                v = src[s * L.cout + o];
            }
            buf[0][sb * ws + o] = v;
        }
    }
    __syncthreads();
    int cur = 0, width = T.first.cout;
#pragma unroll
    for (int l = 0; l < kTailLayers; ++l) {
        if (l >= T.n_rest)
            break;
        const CnnLayerDev &L = T.rest[l];
        if (live && o < L.cout) {
            const float *h = &buf[cur][sb * ws];
            const float *w = L.W + (int64_t)o * width;
            float acc = 0.f;
            for (int k = 0; k < width; ++k)
                acc = fmaf(h[k], w[k], acc);
            const float v = acc + L.b[o];
            buf[cur ^ 1][sb * ws + o] = L.act == HPACML_ACT_RELU ? (v > 0.f ? v : 0.f) : v;
        }
        __syncthreads();
        cur ^= 1;
        width = L.cout;
    }
    if (live && o < width) {
        int64_t p[HPACML_MAX_RANK];
        sweep_point(m, s, p);
        stg(const_cast<float *>(feature_ptr(m, p, interior(m, p), o)), buf[cur][sb * ws + o]);
    }
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
        // [co / 4][ky][kx][ci][co % 4], zero in the padded channels
        d.woff = (int32_t)buf.size();
        buf.resize(buf.size() + (size_t)d.kh * d.kw * CI * CO, 0.f);
        for (int co = 0; co < cout; ++co)
            for (int ci = 0; ci < cin; ++ci)
                for (int ky = 0; ky < d.kh; ++ky)
                    for (int kx = 0; kx < d.kw; ++kx)
                        buf[d.woff + ((((size_t)(co / 4) * d.kh + ky) * d.kw + kx) * CI + ci) * 4 + co % 4] =
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
    // two) whose buffers fit kLdsShared, else one block per CU
    int one = 0;
    for (int ty : {32, 16, 8, 4, 2, 1}) {
        if (ty > 1 && ty / 2 >= H)
            continue;
        FusedArgs a{};
        size_t f0, f1;
        fused_regions(f, ty, &a, &f0, &f1);
        const size_t bytes = (f0 + f1) * sizeof(float);
        if (bytes <= kLdsShared)
            return ty;
        if (!one && bytes <= kLdsOneBlock)
            one = ty;
    }
    return one;
}

hipError_t launch_cnn_fused(const Map32 &in, const Map32 &out, const FeatTable32 *tin, const FeatTable32 *tout,
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
    a.co_last_pad = 4 * f.L[f.n_layers - 1].cout4;
    a.circular = f.circular;
    for (int l = 0; l < f.n_layers; ++l)
        a.L[l] = f.L[l];
    size_t f0, f1;
    fused_regions(f, ty, &a, &f0, &f1);
    a.buf1 = (int32_t)f0;
    for (int l = 0; l <= f.n_layers; ++l) {
        // region sizes stay below 2^16 pixels and widths at most 256 (checked
        // here): the multiply-shift quotient is then exact
        if ((int64_t)a.rh[l] * a.rw[l] >= (1 << 16) || a.rw[l] > 256)
            return hipErrorInvalidValue;
        a.rw_magic[l] = (uint32_t)(((1u << 24) + a.rw[l] - 1) / a.rw[l]);
    }
    const size_t lds = (f0 + f1) * sizeof(float);
    hipError_t e = hipFuncSetAttribute((const void *)cnn_fused_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)lds);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(cnn_fused_kernel, dim3((unsigned)n_tiles), dim3(kThreads), lds, stream, a, f.wts);
    return hipGetLastError();
}

static void divisor(uint32_t d, uint32_t *magic, uint32_t *shift) {
    // i / d == (i * magic) >> (31 + l) for i < 2^31, l = ceil(log2 d), d < 2^31
    int l = 0;
    while ((uint64_t(1) << l) < d)
        ++l;
    *magic = (uint32_t)(((uint64_t(1) << (31 + l)) + d - 1) / d);
    *shift = 31 + l;
}

void cnn_layer_divisors(CnnLayerDev &L) {
    divisor((uint32_t)std::max(L.w2, 1), &L.w2_magic, &L.w2_shift);
    divisor((uint32_t)std::max(L.h2, 1), &L.h2_magic, &L.h2_shift);
}

void cnn_conv_pack(const float *W, int cout, int cin, int kh, int kw, std::vector<float> &dst) {
    const int groups = (cout + kConvG - 1) / kConvG;
    const size_t taps = (size_t)kh * kw * cin, at = dst.size();
    dst.resize(at + groups * taps * kConvG, 0.f);
    for (int co = 0; co < cout; ++co)
        for (int ci = 0; ci < cin; ++ci)
            for (int ky = 0; ky < kh; ++ky)
                for (int kx = 0; kx < kw; ++kx)
                    dst[at + ((co / kConvG) * taps + ((size_t)ky * kw + kx) * cin + ci) * kConvG + co % kConvG] =
                        W[(((size_t)co * cin + ci) * kh + ky) * kw + kx];
}

// Output tile of a fully connected layer: 64 x 64 (4 x 4 outputs per thread,
// two 16-byte LDS reads per 16 FMAs) unless the layer has at most 16
// outputs, where most of such a tile would be padding.
int linear_tile(const CnnLayerDev &L) { return L.cout > 16 ? 64 : 16; }

int linear_splits(const CnnLayerDev &L, int64_t S) {
    if (L.kind != HPACML_LAYER_LINEAR || S <= 0)
        return 1;
    const int64_t K = (int64_t)L.h * L.w * L.cin;
    const int64_t T = linear_tile(L);
    // split products of layers with more than 16 outputs run on the MFMA
    // kernel's 128 x 64 tiles
    const int64_t blocks = T == 64 ? ((S + kMfS - 1) / kMfS) * ((L.cout + kMfO - 1) / kMfO)
                                   : ((S + T - 1) / T) * ((L.cout + T - 1) / T);
    int64_t z = (1024 + blocks - 1) / blocks;                 // about 1024 blocks in all
    z = std::min<int64_t>(z, std::max<int64_t>(1, K / 64));  // at least 64 k per block
    return (int)std::max<int64_t>(1, std::min<int64_t>(z, kLinSplit));
}

// pooled pixels take groups of 2^qshift lanes: windows of at most 16
// positions, so that a group wastes at most 7 of 16 lanes
bool cnn_pool_fusable(const CnnLayerDev &conv, const CnnLayerDev &pool) {
    return conv.kind == HPACML_LAYER_CONV2D && pool.kind == HPACML_LAYER_MAXPOOL2D && pool.sh == pool.kh &&
           pool.sw == pool.kw && pool.kh * pool.kw <= 16;
}

hipError_t launch_cnn_conv(const CnnLayerDev &L, const CnnLayerDev *pool, const float *in, float *out, int64_t S,
                           hipStream_t stream) {
    const int64_t n_pix = S * (pool ? (int64_t)pool->h2 * pool->w2 : (int64_t)L.h2 * L.w2);
    if (n_pix == 0)
        return hipSuccess;
    int qshift = 0;
    while (pool && (1 << qshift) < pool->kh * pool->kw)
        ++qshift;
    const int64_t bx = ((n_pix << qshift) + 255) / 256, by = (L.cout + kConvG - 1) / kConvG;
    if (bx > INT32_MAX || by > 65535)
        return hipErrorInvalidValue;
    if (pool)
        hipLaunchKernelGGL(cnn_conv_kernel<true>, dim3((unsigned)bx, (unsigned)by), dim3(256), 0, stream, L, *pool,
                           qshift, in, out, n_pix);
    else
        hipLaunchKernelGGL(cnn_conv_kernel<false>, dim3((unsigned)bx, (unsigned)by), dim3(256), 0, stream, L, L, 0,
                           in, out, n_pix);
    return hipGetLastError();
}

// Raw split-K partial sums of a fully connected layer into part[splits][S][O]
// (splits >= 2).
hipError_t launch_linear_split(const CnnLayerDev &L, const float *in, float *out, int64_t S, float *part, int splits,
                               hipStream_t stream) {
    const int64_t K = (int64_t)L.h * L.w * L.cin;
    const int64_t Kc = (K + splits - 1) / splits;
    if (linear_tile(L) == 64) {
        const int64_t bx = (S + kMfS - 1) / kMfS, by = (L.cout + kMfO - 1) / kMfO;
        if (bx > INT32_MAX || by > 65535)
            return hipErrorInvalidValue;
        hipLaunchKernelGGL(cnn_linear_mfma_kernel, dim3((unsigned)bx, (unsigned)by, splits), dim3(256), 0, stream, L,
                           in, S, Kc, part);
    } else {
        const int64_t bx = (S + 15) / 16, by = (L.cout + 15) / 16;
        if (bx > INT32_MAX || by > 65535)
            return hipErrorInvalidValue;
        hipLaunchKernelGGL(cnn_linear_kernel<16>, dim3((unsigned)bx, (unsigned)by, splits), dim3(256), 0, stream, L,
                           in, out, S, Kc, part);
    }
    return hipGetLastError();
}

hipError_t launch_cnn_layer(const CnnLayerDev &L, const float *in, float *out, int64_t S, float *part,
                            hipStream_t stream) {
    const int64_t total = S * (int64_t)L.h2 * L.w2 * L.cout;
    if (total == 0)
        return hipSuccess;
    const int64_t blocks = (total + 255) / 256;
    if (blocks > INT32_MAX)
        return hipErrorInvalidValue;
    switch (L.kind) {
    case HPACML_LAYER_CONV2D:
        return launch_cnn_conv(L, nullptr, in, out, S, stream);
    case HPACML_LAYER_MAXPOOL2D:
        hipLaunchKernelGGL(cnn_pool_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, L, in, out, total);
        break;
    default: {
        // K split over up to kLinSplit blocks when the tiles alone leave the
        // chip short of blocks
        const int T = linear_tile(L);
        const int splits = linear_splits(L, S);
        if (splits == 1) {
            const int64_t bx = (S + T - 1) / T, by = (L.cout + T - 1) / T;
            if (bx > INT32_MAX || by > 65535)
                return hipErrorInvalidValue;
            const int64_t K = (int64_t)L.h * L.w * L.cin;
            if (T == 64)
                hipLaunchKernelGGL(cnn_linear_kernel<64>, dim3((unsigned)bx, (unsigned)by, 1), dim3(256), 0, stream,
                                   L, in, out, S, K, part);
            else
                hipLaunchKernelGGL(cnn_linear_kernel<16>, dim3((unsigned)bx, (unsigned)by, 1), dim3(256), 0, stream,
                                   L, in, out, S, K, part);
        } else {
            hipError_t e = launch_linear_split(L, in, out, S, part, splits, stream);
            if (e != hipSuccess)
                return e;
            const int64_t n = S * L.cout;
            hipLaunchKernelGGL(cnn_linear_reduce_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, L,
                               part, out, S, splits);
        }
        break;
    }
    }
    return hipGetLastError();
}

int cnn_tail_start(const std::vector<CnnLayerDev> &ly) {
    const int n = (int)ly.size();
    int t = n;
    // the trailing fully connected layers whose inputs are at most 256 wide
    while (t > 0 && ly[t - 1].kind == HPACML_LAYER_LINEAR && ly[t - 1].cout <= 256 &&
           (int64_t)ly[t - 1].h * ly[t - 1].w * ly[t - 1].cin <= 256)
        --t;
    // the fully connected layer before them (any K) starts the tail
    if (t > 0 && ly[t - 1].kind == HPACML_LAYER_LINEAR && ly[t - 1].cout <= 256)
        --t;
    if (t == n)
        return -1;
    return n - 1 - t <= kTailLayers ? t : -1;
}

hipError_t launch_cnn_tail(const std::vector<CnnLayerDev> &ly, int start, const float *src, int splits,
                           const DevMap &out, int64_t S, hipStream_t stream) {
    if (S == 0)
        return hipSuccess;
    CnnTail T{};
    T.first = ly[start];
    T.n_rest = (int)ly.size() - 1 - start;
    T.splits = splits > 1 ? splits : 0;
    int width = T.first.cout;
    for (int l = 0; l < T.n_rest; ++l) {
        T.rest[l] = ly[start + 1 + l];
        width = std::max(width, T.rest[l].cout);
    }
    int ws = 1;
    while (ws < width)
        ws *= 2;
    T.width = ws;
    const int64_t per = 256 / ws, blocks = (S + per - 1) / per;
    if (blocks > INT32_MAX)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(cnn_tail_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, T, src, out, S);
    return hipGetLastError();
}

hipError_t launch_cnn_linear_partials(const CnnLayerDev &L, const float *in, float *out, int64_t S, float *part,
                                      int *splits, hipStream_t stream) {
    *splits = linear_splits(L, S);
    if (*splits <= 1)
        return launch_cnn_layer(L, in, out, S, part, stream);
    return launch_linear_split(L, in, out, S, part, *splits, stream);
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
