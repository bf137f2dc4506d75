// fp32 fused region kernel: gather -> MLP -> scatter with the activations
// resident in registers and every weight resident in LDS.
//
// The surrogate runs per sweep point on the composed input tensor
// (Sec. IV-A composition, Sec. IV-B inference).  Here each wave owns 32 points
// and computes every layer transposed, H_out^T = W * H_in^T, on
// v_mfma_f32_32x32x2_f32: A = weights (rows = output features, from LDS),
// B = activations (columns = points, from registers), C = the next layer's
// activations.  In the 32x32 C layout lane l holds point l%32 and, in
// register r of m-block mb, feature 32mb + 8(r/4) + 4(l/32) + r%4.  Used
// directly as the next layer's B operand (K-step s takes register s%16 of
// m-block s/16, k = l/32), the activations never leave registers: the next
// layer's weight columns are permuted to match when the LDS image is packed.
//
// First layer: each lane gathers feature 2s + l/32 of its point straight into
// the B operand of K-step s.  Output layer (<= 8 outputs): VALU dot products
// over the lane's 16*NMB features plus one cross-half shuffle.  Biases enter
// as the initial accumulator.
#include "kernels.hpp"

namespace hpacml {

namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
constexpr int kFoutMax = 8;

// LDS image offsets (floats) for a model of hidden width H = 32 * NMB.
struct F32Layout {
    int nmb, ks1, n_hidden, f_out;
    __host__ __device__ int l1() const { return 0; }
    __host__ __device__ int l1_bias() const { return ks1 * 64 * nmb; }
    __host__ __device__ int hidden(int h) const { return l1_bias() + 32 * nmb + h * (32 * nmb * 32 * nmb + 32 * nmb); }
    __host__ __device__ int hidden_bias(int h) const { return hidden(h) + 32 * nmb * 32 * nmb; }
    __host__ __device__ int out_w() const { return hidden(n_hidden); }
    __host__ __device__ int out_b() const { return out_w() + f_out * 32 * nmb; }
    __host__ __device__ int total() const { return out_b() + kFoutMax; }
};

// feature of the previous layer that K-step s, lane half g reads (see above)
__host__ __device__ inline int kperm(int s, int g) {
    return 32 * (s / 16) + 8 * ((s % 16) / 4) + 4 * g + (s % 4);
}
// feature held by lane half g in register r of m-block mb
__host__ __device__ inline int crow(int mb, int r, int g) { return 32 * mb + 8 * (r / 4) + 4 * g + (r % 4); }

template <int NMB>
struct FragA;
template <>
struct FragA<2> {
    float2 v;
    __device__ float operator[](int i) const { return i == 0 ? v.x : v.y; }
};
template <>
struct FragA<4> {
    float4 v;
    __device__ float operator[](int i) const { return i == 0 ? v.x : (i == 1 ? v.y : (i == 2 ? v.z : v.w)); }
};

template <int NMB>
__device__ __forceinline__ FragA<NMB> lds_frag(const float *base, int s, int lane) {
    FragA<NMB> a;
    if constexpr (NMB == 2)
        a.v = reinterpret_cast<const float2 *>(base)[s * 64 + lane];
    else
        a.v = reinterpret_cast<const float4 *>(base)[s * 64 + lane];
    return a;
}

template <int NMB>
__device__ __forceinline__ void load_bias(const float *bias, int g, floatx16 *acc) {
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb) {
        const float4 *p = reinterpret_cast<const float4 *>(bias + (g * NMB + mb) * 16);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            float4 v = p[q];
            acc[mb][4 * q + 0] = v.x;
            acc[mb][4 * q + 1] = v.y;
            acc[mb][4 * q + 2] = v.z;
            acc[mb][4 * q + 3] = v.w;
        }
    }
}

template <int NMB, int KS1MAX, bool PF>
__global__ void __launch_bounds__(512) mlp_f32_kernel(Map32 in, Map32 out, FeatTable32 tin, FeatTable32 tout,
                                                      F32Packed pk, int32_t n_tiles, int32_t xcd_ranges) {
    extern __shared__ float lds[];
    const F32Layout lay{NMB, pk.ks1, pk.n_hidden, pk.f_out};
    const int lane = threadIdx.x & 63;
    const int g = lane >> 5;
    const int col = lane & 31;
    const int waves_per_block = blockDim.x >> 6;
    // XCD-aware order (blocks of one XCD, hardware id % 8, share an L2).
    // Pointwise maps: each round of the grid takes adjacent tiles per XCD.
    // Windowed maps (xcd_ranges, grid a multiple of 8): each XCD walks one
    // contiguous eighth of the tiles, so the rows a window shares with the
    // tiles before it are still in that XCD's L2.
    const int nb = gridDim.x;
    int wave_id, n_waves, t_end;
    if (xcd_ranges) {
        const int per = (n_tiles + 7) / 8;
        const int x = blockIdx.x % 8;
        wave_id = x * per + (blockIdx.x / 8) * waves_per_block + (threadIdx.x >> 6);
        n_waves = (nb / 8) * waves_per_block;
        t_end = (x + 1) * per < n_tiles ? (x + 1) * per : n_tiles;
    } else {
        const int lb = (nb % 8 == 0) ? (blockIdx.x % 8) * (nb / 8) + blockIdx.x / 8 : blockIdx.x;
        wave_id = lb * waves_per_block + (threadIdx.x >> 6);
        n_waves = nb * waves_per_block;
        t_end = n_tiles;
    }
    const int F = in.n_features;

    // ---- gather: lane (col, g) loads feature 2s+g of its point for K-step
    //      s.  The two feature pointers of a K-step come from the kernel
    //      arguments (entries past the last feature repeat it, so the loads
    //      are unconditional and their count fixed); only the dimensions where
    //      the wave touches an edge get a boundary fix-up.  The loads of the
    //      wave's next tile are issued before the current tile's layers run.
    float xn[KS1MAX];
    bool nvalid = false;
    auto gather = [&](int tile) {
        const int b = tile * 32 + col;
        nvalid = b < in.n_points;
        const Pt32 pt = locate32(in, nvalid ? b : in.n_points - 1);
        const uint32_t edge = edge_dims32(in, pt);
#pragma unroll
        for (int s = 0; s < KS1MAX; ++s) {
            const float *p = g ? tin.fptr[2 * s + 1] : tin.fptr[2 * s];
            int32_t idx = pt.pe;
            if (edge)
                idx += edge_fix32(in, pt, g ? tin.raw8[2 * s + 1] : tin.raw8[2 * s], edge);
            // (with PF the load count is fixed, so waiting for this tile's
            // loads never waits for the next tile's)
            xn[s] = (PF || s < pk.ks1) ? ldg(p + idx) : 0.f;
            if (s % 8 == 7)
                __builtin_amdgcn_sched_barrier(0);   // bound the live addresses
        }
    };
    // (without PF -- a wave with a single tile, or the widest variant, which
    // has no registers for a second set -- each tile is gathered just before
    // its use)
    constexpr bool kPrefetch = PF && !(NMB == 4 && KS1MAX == 32);
    // the first tile's loads go out before the weights are staged (their
    // latencies overlap) where registers allow -- H = 64, or at most 16
    // inputs (wider H = 128 variants would spill) -- and, without prefetch,
    // when it is the wave's only tile
    constexpr bool kEarly = NMB == 2 || KS1MAX <= 8;
    bool gathered = false;
    if (kEarly && wave_id < t_end && (kPrefetch || wave_id + n_waves >= t_end)) {
        gather(wave_id);
        gathered = true;
    }

    // stage the packed weights once per block
    {
        const float4 *src = reinterpret_cast<const float4 *>(pk.image);
        float4 *dstl = reinterpret_cast<float4 *>(lds);
        const int n4 = pk.lds_bytes / 16;
        for (int i = threadIdx.x; i < n4; i += blockDim.x)
            dstl[i] = src[i];
    }
    __syncthreads();
    if (kPrefetch && !gathered && wave_id < t_end)
        gather(wave_id);

    for (int tile = wave_id; tile < t_end; tile += n_waves) {
        const int b = tile * 32 + col;
        if (!kPrefetch && !gathered)
            gather(tile);
        gathered = false;
        const bool valid = nvalid;
        float x[KS1MAX];
#pragma unroll
        for (int s = 0; s < KS1MAX; ++s)
            x[s] = xn[s];
        if (kPrefetch)
            gather(tile + n_waves < t_end ? tile + n_waves : tile);
#pragma unroll
        for (int s = 0; s < KS1MAX; ++s)
            x[s] = (valid && 2 * s + g < F) ? x[s] : 0.f;

        floatx16 acc[NMB];
        // ---- first layer: K = 2 * ks1 (zero-padded features)
        load_bias<NMB>(lds + lay.l1_bias(), g, acc);
#pragma unroll
        for (int s = 0; s < KS1MAX; ++s) {
            if (s < pk.ks1) {
                FragA<NMB> a = lds_frag<NMB>(lds + lay.l1(), s, lane);
#pragma unroll
                for (int mb = 0; mb < NMB; ++mb)
                    acc[mb] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[mb], x[s], acc[mb], 0, 0, 0);
            }
        }
        if (pk.act[0] == HPACML_ACT_RELU) {
#pragma unroll
            for (int mb = 0; mb < NMB; ++mb)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    acc[mb][r] = relu_mfma(acc[mb][r]);
        }

        // ---- hidden layers H -> H
        for (int h = 0; h < pk.n_hidden; ++h) {
            floatx16 hin[NMB];
#pragma unroll
            for (int mb = 0; mb < NMB; ++mb)
                hin[mb] = acc[mb];
            load_bias<NMB>(lds + lay.hidden_bias(h), g, acc);
            const float *wl = lds + lay.hidden(h);
#pragma unroll
            for (int s = 0; s < 16 * NMB; ++s) {
                FragA<NMB> a = lds_frag<NMB>(wl, s, lane);
                const float bv = hin[s / 16][s % 16];
#pragma unroll
                for (int mb = 0; mb < NMB; ++mb)
                    acc[mb] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[mb], bv, acc[mb], 0, 0, 0);
            }
            if (pk.act[h + 1] == HPACML_ACT_RELU) {
#pragma unroll
                for (int mb = 0; mb < NMB; ++mb)
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        acc[mb][r] = relu_mfma(acc[mb][r]);
            }
        }

        // ---- output layer (VALU) + scatter through the `from` map
        const Pt32 po = locate32(out, valid ? b : in.n_points - 1);
        const uint32_t oedge = edge_dims32(out, po);
        const bool orelu = pk.act[pk.n_hidden + 1] == HPACML_ACT_RELU;
        for (int go = 0; go < pk.f_out; ++go) {
            const float *w = lds + lay.out_w() + (go * 2 + g) * (16 * NMB);
            float part = 0.f;
#pragma unroll
            for (int mb = 0; mb < NMB; ++mb)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const float4 wv = reinterpret_cast<const float4 *>(w + mb * 16)[q];
                    part = fmaf(acc[mb][4 * q + 0], wv.x, part);
                    part = fmaf(acc[mb][4 * q + 1], wv.y, part);
                    part = fmaf(acc[mb][4 * q + 2], wv.z, part);
                    part = fmaf(acc[mb][4 * q + 3], wv.w, part);
                }
            part += __shfl_xor(part, 32);
            float y = part + lds[lay.out_b() + go];
            if (orelu)
                y = fmaxf(y, 0.f);
            if (g == 0 && valid)
                stg(const_cast<float *>(tout.fptr[go]) + (po.pe + (oedge ? edge_fix32(out, po, tout.raw8[go], oedge) : 0)), y);
        }
    }
}

template <int NMB, int KS1MAX>
hipError_t launch_t(const Map32 &in, const Map32 &out, const FeatTable32 &tin, const FeatTable32 &tout,
                    const F32Packed &pk, hipStream_t stream) {
    const int32_t n_tiles = (in.n_points + 31) / 32;
    const int threads = NMB == 4 ? 512 : 256;
    const int waves = threads / 64;
    const size_t lds = (size_t)pk.lds_bytes;
    int per_cu = (int)(163840 / (lds + 1024));
    per_cu = per_cu < 1 ? 1 : (per_cu > 4 ? 4 : per_cu);
    int64_t grid = 256LL * per_cu;
    const int64_t need = (n_tiles + waves - 1) / waves;
    if (grid > need)
        grid = need;
    // windowed maps: one contiguous range of tiles per XCD (see the kernel)
    bool window = false;
    for (int d = 0; d < in.rank; ++d)
        window = window || in.omin[d] != 0 || in.omax[d] != 0;
    const int32_t xcd_ranges = window && grid % 8 == 0;
    // prefetch only when waves take more than one tile
    const int64_t per_wave = xcd_ranges ? (n_tiles + 7) / 8 : n_tiles, waves_each = xcd_ranges ? grid / 8 * waves : grid * waves;
    auto kern = per_wave > waves_each ? mlp_f32_kernel<NMB, KS1MAX, true> : mlp_f32_kernel<NMB, KS1MAX, false>;
    hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(threads), lds, stream, in, out, tin, tout, pk, n_tiles,
                       xcd_ranges);
    return hipGetLastError();
}

}  // namespace

bool f32_fast_supported(int n_layers, const int32_t *dims, int compute) {
    if (compute != HPACML_F32 || n_layers < 2 || n_layers > HPACML_MAX_LAYERS)
        return false;
    const int H = dims[1];
    if (H != 64 && H != 128)
        return false;
    for (int l = 1; l < n_layers; ++l)
        if (dims[l] != H)
            return false;
    if (dims[0] > 64 || dims[n_layers] > kFoutMax)
        return false;
    return f32_image_floats(n_layers, dims) * 4 <= 150 * 1024;
}

size_t f32_image_floats(int n_layers, const int32_t *dims) {
    F32Layout lay{dims[1] / 32, (dims[0] + 1) / 2, n_layers - 2, dims[n_layers]};
    size_t n = (size_t)lay.total();
    return (n + 3) & ~size_t(3);
}

// Host packing of the LDS image (see F32Layout): A fragments in the order the
// lanes read them, biases and output weights in the C-fragment order.
void f32_pack(int n_layers, const int32_t *dims, const float *const *W, const float *const *b,
              float *img) {
    const int H = dims[1], NMB = H / 32, Fin = dims[0], Fout = dims[n_layers];
    F32Layout lay{NMB, (Fin + 1) / 2, n_layers - 2, Fout};
    for (int i = 0; i < lay.total(); ++i)
        img[i] = 0.f;
    auto put_bias = [&](int off, const float *bias) {
        for (int g = 0; g < 2; ++g)
            for (int mb = 0; mb < NMB; ++mb)
                for (int r = 0; r < 16; ++r)
                    img[off + (g * NMB + mb) * 16 + r] = bias[crow(mb, r, g)];
    };
    // first layer: K-step s, lane l -> W1[32mb + l%32][2s + l/32]
    for (int s = 0; s < lay.ks1; ++s)
        for (int l = 0; l < 64; ++l)
            for (int mb = 0; mb < NMB; ++mb) {
                const int k = 2 * s + l / 32, o = 32 * mb + l % 32;
                img[lay.l1() + (s * 64 + l) * NMB + mb] = k < Fin ? W[0][(size_t)o * Fin + k] : 0.f;
            }
    put_bias(lay.l1_bias(), b[0]);
    for (int h = 0; h < lay.n_hidden; ++h) {
        const float *Wh = W[h + 1];
        for (int s = 0; s < 16 * NMB; ++s)
            for (int l = 0; l < 64; ++l)
                for (int mb = 0; mb < NMB; ++mb) {
                    const int k = kperm(s, l / 32), o = 32 * mb + l % 32;
                    img[lay.hidden(h) + (s * 64 + l) * NMB + mb] = Wh[(size_t)o * H + k];
                }
        put_bias(lay.hidden_bias(h), b[h + 1]);
    }
    const float *Wo = W[n_layers - 1];
    for (int go = 0; go < Fout; ++go)
        for (int g = 0; g < 2; ++g)
            for (int mb = 0; mb < NMB; ++mb)
                for (int r = 0; r < 16; ++r)
                    img[lay.out_w() + (go * 2 + g) * 16 * NMB + mb * 16 + r] =
                        Wo[(size_t)go * H + crow(mb, r, g)];
    for (int go = 0; go < Fout; ++go)
        img[lay.out_b() + go] = b[n_layers - 1][go];
}

hipError_t launch_mlp_f32(const Map32 &in, const Map32 &out, const FeatTable32 &tin, const FeatTable32 &tout,
                          const F32Packed &pk, hipStream_t stream) {
    if (in.n_points == 0)
        return hipSuccess;
    if (pk.hid == 128)
        return pk.ks1 <= 8 ? launch_t<4, 8>(in, out, tin, tout, pk, stream)
                           : (pk.ks1 <= 20 ? launch_t<4, 20>(in, out, tin, tout, pk, stream)
                                           : launch_t<4, 32>(in, out, tin, tout, pk, stream));
    return pk.ks1 <= 8 ? launch_t<2, 8>(in, out, tin, tout, pk, stream)
                       : (pk.ks1 <= 20 ? launch_t<2, 20>(in, out, tin, tout, pk, stream)
                                       : launch_t<2, 32>(in, out, tin, tout, pk, stream));
}

const char *f32_variant_name(const F32Packed &pk) {
    if (pk.hid == 128)
        return pk.ks1 <= 8 ? "mlp_f32_h128_k16" : (pk.ks1 <= 20 ? "mlp_f32_h128_k40" : "mlp_f32_h128_k64");
    return pk.ks1 <= 8 ? "mlp_f32_h64_k16" : (pk.ks1 <= 20 ? "mlp_f32_h64_k40" : "mlp_f32_h64_k64");
}

}  // namespace hpacml
