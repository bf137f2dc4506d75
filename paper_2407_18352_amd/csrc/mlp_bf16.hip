// bf16 fused region kernel: gather -> MLP -> scatter for wide hidden layers
// (H in {256, 512}), bf16 operands with fp32 accumulation on
// v_mfma_f32_32x32x16_bf16 (first and hidden layers) and
// v_mfma_f32_16x16x32_bf16 (output layer).
//
// The surrogate runs per sweep point on the composed input tensor
// (Sec. IV-A composition, Sec. IV-B inference).  The hidden weights of these
// models (128 KB - 512 KB per layer in bf16) do not fit in LDS, so the roles
// are the reverse of the fp32 kernel: a block of 8 waves (2 per SIMD) owns a
// tile of T points (T * H = 65536) whose activations sit in LDS as bf16
// [T][H] (128 KB), and the weights stream from L2 straight into MFMA A
// fragments (prepacked so each fragment is one 16-byte load per lane).  Every
// layer is H_out^T = W * H_in^T; each wave computes a 64-feature x 128-point
// block, so each weight fragment fetched from L2 feeds 4 MFMAs and each
// activation fragment read from LDS feeds 2.  Per layer: the K loop (A from
// L2, B from LDS) into 128 fp32 accumulators per lane, a block barrier, then
// the epilogue applies the activation, rounds to bf16 and stores over the
// layer's input.
//
// Biases ride in the K dimension: each activation row carries a constant
// chunk [1, 1, 1, 0, ...] and the weight fragments of one extra K-step hold
// the fp32 bias split exactly into three bf16 terms (hi + mid + lo), so the
// MFMA accumulates the bias and the epilogue is activation + conversion only.
// The first layer uses spare columns of its zero-padded K the same way.
//
// LDS rows are sequences of 16-byte chunks (8 bf16).  The epilogue stores the
// 16 values a lane holds for one (m-block, point) as two chunks; the order of
// features inside a chunk is fixed by the MFMA C layout, and the next layer's
// weight columns are permuted to match when the weights are packed.  Rows are
// padded to an odd number of chunks, so the 8 lanes (8 consecutive points)
// that share an LDS cycle hit distinct banks, and every address is a per-lane
// base plus a compile-time offset.
#include "kernels.hpp"

namespace hpacml {

namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kThreads = 512;   // 8 waves, 2 per SIMD

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

// Raw buffer view of the packed weights: loads take a per-lane byte offset
// plus a wave-uniform offset, so the K loop keeps no per-step 64-bit
// addresses in VGPRs; accesses past `bytes` read zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t weight_rsrc(const void *p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ uint4 wload(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}

// two fp32 -> packed bf16 pair (round to nearest even), one instruction
__device__ __forceinline__ uint32_t pack2(float a, float b) {
    const floatx2 v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

__device__ __forceinline__ uint4 pack8(const float *v) {
    uint4 q;
    q.x = pack2(v[0], v[1]);
    q.y = pack2(v[2], v[3]);
    q.z = pack2(v[4], v[5]);
    q.w = pack2(v[6], v[7]);
    return q;
}


// feature held at element e of LDS chunk c (C layout of the 32x32 MFMA,
// two chunks per (m-block, lane half))
__host__ __device__ inline int chunk_feature(int c, int e) {
    return 32 * (c / 4) + 16 * ((c % 4) / 2) + 8 * (e / 4) + 4 * (c % 2) + (e % 4);
}

// Tile geometry: 8 waves in a WM x WN grid; every wave computes a 64-feature
// x 128-point block (2 x 4 MFMA blocks, 128 fp32 accumulators per lane).
template <int H>
struct Geo {
    static constexpr int T = 65536 / H;          // points per tile
    static constexpr int NMB = H / 32;           // 32-row m-blocks per layer
    static constexpr int WM = H / 64;            // waves along features
    static constexpr int WN = 8 / WM;            // waves along points
    static constexpr int KS = H / 16;            // K-steps of a hidden layer (plus one for the bias)
    static constexpr int RC = H / 8;             // chunks of activations per row
    static constexpr int PH = RC + 3;            // row pitch: activations, bias chunk, zero chunk, pad
    static constexpr int NB16 = T / 128;         // 16-point n-blocks per wave (output layer)
    static_assert(T / WN == 128, "wave tile is 128 points");
};

template <int H, int KS1MAX>
__global__ void __launch_bounds__(kThreads) mlp_bf16_kernel(Map32 in, Map32 out, FeatTable32 tin, FeatTable32 tout, BF16Packed pk,
                                                            int32_t n_tiles) {
    using G = Geo<H>;
    constexpr int KO = H / 32;                     // output-layer K-steps
    extern __shared__ uint4 smem[];
    uint4 *Hs = smem;                              // [T][PH] activations
    // gathered inputs [T][2 KS1MAX] in the first chunks of each activation row:
    // a row's activations are dead from the previous tile's output layer
    // until the first layer's epilogue, which comes after the first layer
    // has read them
    uint4 *Xs = smem;
    constexpr int XP = G::PH;                      // Xs row pitch
    uint4 *Wo = smem + G::T * G::PH;               // [KO][64] output-layer fragments, staged once
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = tid >> 6;
    const int wm = w % G::WM, wn = w / G::WM;
    const int g = lane >> 5;
    const int col = lane & 31;
    const int m0 = 2 * wm;                         // first m-block of this wave
    const int p0 = 128 * wn + col;                 // this lane's point in n-block 0
    const int F = in.n_features;
    const int nchunk_in = 2 * pk.ks1;              // chunks the first layer reads
    const __amdgpu_buffer_rsrc_t wr = weight_rsrc(pk.frags, pk.frag_bytes);
    const uint32_t vlane = (uint32_t)((m0 * 64 + lane) * 16);

    __shared__ const float *so_ptr[16];             // output table and biases, F_out <= 16
    __shared__ uint32_t so_raw[16];
    __shared__ float so_bias[16];
    if (tid < 16) {
        so_ptr[tid] = tout.fptr[tid];
        so_raw[tid] = tout.raw8[tid];
        so_bias[tid] = pk.bias_out[tid];
    }
    // output-layer fragments, the same for every tile
    for (int k = tid; k < KO * 64; k += kThreads)
        Wo[k] = wload(weight_rsrc(pk.frags, pk.frag_bytes), (uint32_t)(k * 16), (uint32_t)(pk.off_wo * 16));
    // constant chunks of every activation row: [1,1,1,0,...] then zeros
    for (int r = tid; r < G::T; r += kThreads) {
        const float one3[8] = {1.f, 1.f, 1.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        Hs[r * G::PH + G::RC] = pack8(one3);
        Hs[r * G::PH + G::RC + 1] = uint4{0u, 0u, 0u, 0u};
    }
    __syncthreads();

    // XCD-aware tile order: blocks on one XCD take adjacent tiles
    const int nb = gridDim.x;
    const int lb = (nb % 8 == 0) ? (blockIdx.x % 8) * (nb / 8) + blockIdx.x / 8 : blockIdx.x;

    // scatter through the `from` map: lane (l%16 = point, l/16 = output
    // group) of wave w holds outputs 4(l/16)..+3 of point w*T/8 + 16n + l%16
    const bool orelu = pk.act[pk.n_hidden + 1] == HPACML_ACT_RELU;
    // the output index varies across a wave here: its table entries and
    // bias are read from an LDS copy (an indexed kernel argument would be a
    // vector load, and waiting for it would also wait for the next tile's
    // gather loads issued before it)
    auto scatter = [&](int bs, const floatx4 *y) {
        const int q = lane >> 4, pc = lane & 15;
#pragma unroll
        for (int n = 0; n < G::NB16; ++n) {
            const int b = bs + w * (G::T / 8) + 16 * n + pc;
            const Pt32 pt = locate32(out, b < out.n_points ? b : out.n_points - 1);
            const uint32_t edge = edge_dims32(out, pt);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int go = 4 * q + r;
                if (go < pk.f_out && b < out.n_points) {
                    float v = y[n][r] + so_bias[go];
                    if (orelu)
                        v = fmaxf(v, 0.f);
                    int32_t idx = pt.pe;
                    if (edge)
                        idx += edge_fix32(out, pt, so_raw[go], edge);
                    stg(const_cast<float *>(so_ptr[go]) + idx, v);
                }
            }
        }
    };

    // ---- gather: (point, chunk) pairs, 8 features per chunk, rounded to
    //      bf16; features F..F+2 are the constant 1 that carries the
    //      first-layer bias.  Every pass of a thread has the same point (the
    //      block size is a multiple of T), so its sweep point is resolved
    //      once; T is a multiple of 64, so the chunk is wave-uniform and its
    //      eight feature pointers come from the kernel arguments.  Loads are
    //      unconditional (table entries past the last feature repeat it;
    //      unused values are replaced when stored), so all of them are in
    //      flight before the first use; only the dimensions where the wave
    //      touches an edge get a boundary fix-up.  The loads of tile t+1 are
    //      issued after the first layer of tile t and land in registers.
    constexpr int PASSES = (G::T * 2 * KS1MAX + kThreads - 1) / kThreads;
    const int gp = tid % G::T;                     // this thread's point in a tile
    float gv[PASSES][8];
    bool gvalid = false;
    auto gather_issue = [&](int tile) {
        const int b = tile * G::T + gp;
        gvalid = b < in.n_points;
        const Pt32 pt = locate32(in, gvalid ? b : in.n_points - 1);
        const uint32_t edge = edge_dims32(in, pt);
#pragma unroll
        for (int it = 0; it < PASSES; ++it) {
            int c = __builtin_amdgcn_readfirstlane((tid + it * kThreads) / G::T);
            c = c < nchunk_in ? c : nchunk_in - 1;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                int32_t idx = pt.pe;
                if (edge)
                    idx += edge_fix32(in, pt, tin.raw8[8 * c + e], edge);
                gv[it][e] = ldg(tin.fptr[8 * c + e] + idx);
            }
        }
    };
    // first-layer weight fragments (the same for every tile), reloaded for
    // each tile where registers are free: before the last epilogue of the
    // previous tile, so their latency hides behind it
    uint4 a1[KS1MAX][2];
    auto load_a1 = [&]() {
#pragma unroll
        for (int s = 0; s < KS1MAX; ++s)
#pragma unroll
            for (int j = 0; j < 2; ++j)
                a1[s][j] = s < pk.ks1 ? wload(wr, vlane + j * 1024, (uint32_t)((pk.off_w1 + (int64_t)s * G::NMB * 64) * 16))
                                      : uint4{0u, 0u, 0u, 0u};
    };
    // 3-D windows with whole tiles per row: z fastest in the visit order, so
    // the blocks of one XCD take consecutive planes of one column of tiles
    // and the plane neighbours a tile reads are the tiles beside it in time
    // (plane-strided addresses otherwise collide in the caches: 1.7% faster
    // on the 512^3 grid)
    const bool zorder = in.rank == 3 && in.count[2] % G::T == 0 && in.omin[0] != in.omax[0];
    const int nz = in.count[0];
    const int per_plane = zorder ? n_tiles / nz : 1;
    auto tile_of = [&](int u) { return zorder ? (u % nz) * per_plane + u / nz : u; };
    if (lb < n_tiles) {
        gather_issue(tile_of(lb));
        load_a1();
    }

    for (int u = lb; u < n_tiles; u += nb) {
        const int tile = tile_of(u);
        const int b0 = tile * G::T;

        __syncthreads();                               // the previous tile's output layer is done with Hs
#pragma unroll
        for (int it = 0; it < PASSES; ++it) {
            const int c = __builtin_amdgcn_readfirstlane((tid + it * kThreads) / G::T);
            float u[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int f = 8 * c + e;
                u[e] = f < F ? (gvalid ? gv[it][e] : 0.f) : (f < F + 3 ? 1.f : 0.f);
            }
            if (c < nchunk_in)
                Xs[gp * XP + c] = pack8(u);
        }
        __syncthreads();

        floatx16 acc[2][4];

        // ---- first layer: A = W1 fragments (bias in columns F..F+2), B =
        //      gathered inputs (LDS); accumulators start from zero
#pragma unroll
        for (int s = 0; s < KS1MAX; ++s) {
            if (s < pk.ks1) {
#pragma unroll
                for (int n = 0; n < 4; ++n) {
                    const bf16x8 bv = as_bf16x8(Xs[(p0 + 32 * n) * XP + 2 * s + g]);
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        acc[j][n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                            as_bf16x8(a1[s][j]), bv, s == 0 ? floatx16{} : acc[j][n], 0, 0, 0);
                }
            }
        }

        // ---- hidden layers: epilogue of the previous layer (activation,
        //      bf16 into LDS), then H x H plus the bias K-step.  The first
        //      weight fragments of what follows (the next hidden layer, or the
        //      output layer) are requested before the epilogue so their L2
        //      latency hides behind it.
        constexpr int KT = G::KS + 1;
        // epilogue of layer h's accumulators: activation, bf16, into Hs
        auto epilogue = [&](int h) {
            __syncthreads();               // every wave is done reading Hs (and Xs)
            if (pk.act[h] == HPACML_ACT_RELU) {
#pragma unroll
                for (int j = 0; j < 2; ++j)
#pragma unroll
                    for (int n = 0; n < 4; ++n)
#pragma unroll
                        for (int sp = 0; sp < 2; ++sp) {
                            float v[8];
#pragma unroll
                            for (int e = 0; e < 8; ++e)
                                v[e] = relu_mfma(acc[j][n][8 * sp + e]);
                            Hs[(p0 + 32 * n) * G::PH + 4 * (m0 + j) + 2 * sp + g] = pack8(v);
                        }
            } else {
#pragma unroll
                for (int j = 0; j < 2; ++j)
#pragma unroll
                    for (int n = 0; n < 4; ++n)
#pragma unroll
                        for (int sp = 0; sp < 2; ++sp) {
                            float v[8];
#pragma unroll
                            for (int e = 0; e < 8; ++e)
                                v[e] = acc[j][n][8 * sp + e];
                            Hs[(p0 + 32 * n) * G::PH + 4 * (m0 + j) + 2 * sp + g] = pack8(v);
                        }
            }
            __syncthreads();               // the layer's activations are complete
        };

        // the next tile's gather loads (the last tile re-reads itself, so the
        // issue is unconditional) land during the hidden layers, the last
        // epilogue and the output layer: windowed maps read neighbouring rows
        // and planes that often miss the L2, and a shorter lead left part of
        // that latency exposed
        gather_issue(tile_of(u + nb < n_tiles ? u + nb : u));
        uint4 A[4][2];
        for (int h = 0; h < pk.n_hidden; ++h) {
            const uint32_t wbase = (uint32_t)((pk.off_wh + (int64_t)h * KT * G::NMB * 64) * 16);
            auto load_a = [&](uint4 *dst, int s) {
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    dst[j] = wload(wr, vlane + j * 1024, wbase + (uint32_t)s * G::NMB * 1024);
            };
            load_a(A[0], 0);
            load_a(A[1], 1);
            load_a(A[2], 2);
            epilogue(h);

            // K loop, fully unrolled; scheduling barriers pin the pipeline:
            // weight fragments three K-steps ahead (ring of 4), activation
            // fragments one K-step ahead (ring of 2)
            uint4 Bq[2][4];
            auto load_b = [&](uint4 *dst, int s) {
#pragma unroll
                for (int n = 0; n < 4; ++n)
                    dst[n] = Hs[(p0 + 32 * n) * G::PH + 2 * s + g];
            };
            load_b(Bq[0], 0);
#pragma unroll
            for (int s = 0; s < KT; ++s) {
                if (s + 3 < KT)
                    load_a(A[(s + 3) & 3], s + 3);
                if (s + 1 < KT)
                    load_b(Bq[(s + 1) & 1], s + 1);
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int n = 0; n < 4; ++n) {
                    const bf16x8 bv = as_bf16x8(Bq[s & 1][n]);
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        acc[j][n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                            as_bf16x8(A[s & 3][j]), bv, s == 0 ? floatx16{} : acc[j][n], 0, 0, 0);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        load_a1();
        epilogue(pk.n_hidden);

        // ---- output layer: 16 x T, K = H on 16x16x32; wave w takes points
        //      [w*T/8, (w+1)*T/8); lane (l%16 = point, l/16 = k group)
        {
            const int q = lane >> 4, pc = lane & 15;
            floatx4 y[G::NB16];
#pragma unroll
            for (int s = 0; s < KO; ++s) {
                const bf16x8 av = as_bf16x8(Wo[s * 64 + lane]);
#pragma unroll
                for (int n = 0; n < G::NB16; ++n) {
                    const int p = w * (G::T / 8) + 16 * n + pc;
                    const bf16x8 bv = as_bf16x8(Hs[p * G::PH + 4 * s + q]);
                    y[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, s == 0 ? floatx4{} : y[n], 0, 0, 0);
                }
            }
            scatter(b0, y);
        }
        // the next tile's gather stores to Xs after a barrier; Hs is not
        // written again before a barrier
    }
}

template <int H, int KS1MAX>
hipError_t launch_t(const Map32 &in, const Map32 &out, const FeatTable32 &tin, const FeatTable32 &tout,
                    const BF16Packed &pk, hipStream_t stream) {
    using G = Geo<H>;
    const int32_t n_tiles = (in.n_points + G::T - 1) / G::T;
    static_assert(2 * KS1MAX + 1 <= G::RC, "gathered inputs fit in an activation row");
    const size_t lds = (size_t)G::T * G::PH * 16 + (size_t)(H / 32) * 64 * 16;
    const int32_t grid = n_tiles < 256 ? n_tiles : 256;
    auto kern = mlp_bf16_kernel<H, KS1MAX>;
    hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kThreads), lds, stream, in, out, tin, tout, pk, n_tiles);
    return hipGetLastError();
}

}  // namespace

uint16_t bf16_rne_host(float x) {
    uint32_t u;
    std::memcpy(&u, &x, 4);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u)
        return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

float bf16_value(uint16_t h) {
    const uint32_t u = (uint32_t)h << 16;
    float f;
    std::memcpy(&f, &u, 4);
    return f;
}

// fp32 bias as three bf16 terms with hi + mid + lo == b exactly: hi and mid
// keep the leading 8 significant bits of b and of b - hi (truncation, so the
// differences stay exact), lo the last 8.
void split_bias(float b, uint16_t out[3]) {
    uint32_t u;
    std::memcpy(&u, &b, 4);
    out[0] = (uint16_t)(u >> 16);
    const float r1 = b - bf16_value(out[0]);
    std::memcpy(&u, &r1, 4);
    out[1] = (uint16_t)(u >> 16);
    const float r2 = r1 - bf16_value(out[1]);
    out[2] = bf16_rne_host(r2);
}

bool bf16_fast_supported(int n_layers, const int32_t *dims, int compute) {
    if (compute != HPACML_BF16 || n_layers < 2 || n_layers > HPACML_MAX_LAYERS)
        return false;
    const int H = dims[1];
    if (H != 256 && H != 512)
        return false;
    for (int l = 1; l < n_layers; ++l)
        if (dims[l] != H)
            return false;
    // the gathered-input rows (F_in + 3 bias columns) share the 160 KB of LDS
    // with the activations
    return dims[0] + 3 <= (H == 512 ? 64 : 16) && dims[n_layers] <= 16;
}

// Packed layout (uint16 units):
//   W1 fragments [ks1][NMB][64 lanes][8]      A[i=l%32][k=8(l/32)+e] = W1[32m+i][16s+k];
//                                             columns F..F+2 hold the bias terms
//   hidden       [n_hidden][KS+1][NMB][64][8] columns permuted to the LDS chunk
//                                             order; K-step KS holds the bias terms
//   output       [H/32][64][8]                A[i=l%16][k=8(l/16)+e] (16x16x32 layout)
size_t bf16_pack(int n_layers, const int32_t *dims, const float *const *W, const float *const *b,
                 std::vector<uint16_t> &frags, BF16Packed *pk) {
    const int H = dims[1], Fin = dims[0], Fout = dims[n_layers];
    const int NMB = H / 32, KS = H / 16, ks1 = (Fin + 3 + 15) / 16;
    const int n_hidden = n_layers - 2;
    frags.clear();
    pk->off_w1 = 0;
    for (int s = 0; s < ks1; ++s)
        for (int m = 0; m < NMB; ++m)
            for (int l = 0; l < 64; ++l)
                for (int e = 0; e < 8; ++e) {
                    const int o = 32 * m + l % 32, k = 16 * s + 8 * (l / 32) + e;
                    uint16_t v = 0;
                    if (k < Fin) {
                        v = bf16_rne_host(W[0][(size_t)o * Fin + k]);
                    } else if (k < Fin + 3) {
                        uint16_t t[3];
                        split_bias(b[0][o], t);
                        v = t[k - Fin];
                    }
                    frags.push_back(v);
                }
    pk->off_wh = (int64_t)(frags.size() / 8);
    for (int h = 0; h < n_hidden; ++h)
        for (int s = 0; s <= KS; ++s)
            for (int m = 0; m < NMB; ++m)
                for (int l = 0; l < 64; ++l)
                    for (int e = 0; e < 8; ++e) {
                        const int o = 32 * m + l % 32;
                        uint16_t v = 0;
                        if (s < KS) {
                            const int k = chunk_feature(2 * s + l / 32, e);
                            v = bf16_rne_host(W[h + 1][(size_t)o * H + k]);
                        } else if (l / 32 == 0 && e < 3) {
                            uint16_t t[3];
                            split_bias(b[h + 1][o], t);
                            v = t[e];
                        }
                        frags.push_back(v);
                    }
    pk->off_wo = (int64_t)(frags.size() / 8);
    for (int s = 0; s < H / 32; ++s)
        for (int l = 0; l < 64; ++l)
            for (int e = 0; e < 8; ++e) {
                const int i = l % 16;
                const int k = chunk_feature(4 * s + l / 16, e);
                frags.push_back(i < Fout ? bf16_rne_host(W[n_layers - 1][(size_t)i * H + k]) : 0);
            }
    pk->frag_bytes = (uint32_t)(frags.size() * 2);
    pk->hid = H;
    pk->n_hidden = n_hidden;
    pk->ks1 = ks1;
    pk->f_out = Fout;
    for (int i = 0; i < 16; ++i)
        pk->bias_out[i] = i < Fout ? b[n_layers - 1][i] : 0.f;
    return frags.size();
}

hipError_t launch_mlp_bf16(const Map32 &in, const Map32 &out, const FeatTable32 &tin, const FeatTable32 &tout,
                           const BF16Packed &pk, hipStream_t stream) {
    if (in.n_points == 0)
        return hipSuccess;
    if (pk.hid == 512)
        return pk.ks1 <= 1 ? launch_t<512, 1>(in, out, tin, tout, pk, stream)
                           : (pk.ks1 <= 3 ? launch_t<512, 3>(in, out, tin, tout, pk, stream)
                                          : launch_t<512, 4>(in, out, tin, tout, pk, stream));
    return launch_t<256, 1>(in, out, tin, tout, pk, stream);
}

const char *bf16_variant_name(const BF16Packed &pk) {
    return pk.hid == 512 ? "mlp_bf16_h512" : "mlp_bf16_h256";
}

}  // namespace hpacml
