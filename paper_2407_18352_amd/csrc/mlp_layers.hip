// Layer-by-layer MLP inference (Sec. IV-B: the surrogate is a stack of
// Linear/ReLU layers evaluated on the gathered input tensor) for shapes no
// fused kernel takes, even with its hidden layers zero-padded: hidden widths
// above 512 (bf16) or 128 (fp32), more hidden layers, inputs or outputs than
// a kernel's limits, and maps outside the 32-bit form.
//
// A chunk of points goes through the layers in turn; activations live in
// two buffers as rows of bf16 (bf16 models) or fp32, one row per point.
//   - First layer: when its input width is small (the usual surrogate: a few
//     physical inputs into a wide layer) one kernel gathers the inputs and
//     computes the layer on the vector ALU, each thread holding the weights
//     of 8 (bf16) or 4 (fp32) neurons in registers and storing 16 bytes per
//     point; otherwise a gather kernel writes the input rows and the layer
//     is a matmul like the others.
//   - Middle layers: one hipBLASLt matmul each, column-major
//     D[N x C] = W[N x K] X[K x C], the bias and the activation (ReLU or
//     identity) applied to the fp32 accumulators in its epilogue.
//   - Last layer: with at most 8 outputs, one kernel computes it (8 lanes
//     per point over 128-byte row segments, a shuffle reduction) and writes
//     the outputs through the `from` map; otherwise a matmul into fp32 rows
//     and a scatter kernel.
// Hidden activations of a bf16 model are rounded to bf16 (nearest-even),
// outputs stay fp32: the rounding points of the fused kernels.  Points are
// processed in chunks of about 1 GB of activations per buffer.
#include <hipblaslt/hipblaslt.h>

#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <vector>

#include "layers.hpp"

namespace hpacml {

namespace {

constexpr int kMaxDevices = 64;
constexpr size_t kLibWorkspace = (size_t)64 << 20;   // the library's scratch, per chunk matmul
constexpr int kCandidates = 8;                         // algorithms asked of the library's heuristic
constexpr int kFirstMaxK = 12;     // input widths the fused gather + first-layer kernel takes
constexpr int kLastMaxOut = 8;     // output counts the fused last-layer + scatter kernel takes
constexpr int kLastMaxK = 1024;    // and input widths (its weights in LDS)
constexpr int kTileP = 64;         // points per tile of the first-layer kernel

// One library handle per device, created on first use and kept for the
// life of the process (handles are not freed while other models may use them).
std::mutex g_lt_mu;
hipblasLtHandle_t g_lt[kMaxDevices] = {};

hipblasLtHandle_t lt_handle(int device) {
    if (device < 0 || device >= kMaxDevices)
        return nullptr;
    std::lock_guard<std::mutex> lock(g_lt_mu);
    if (!g_lt[device]) {
        hipblasLtHandle_t h = nullptr;
        if (hipblasLtCreate(&h) != HIPBLAS_STATUS_SUCCESS)
            return nullptr;
        g_lt[device] = h;
    }
    return g_lt[device];
}

hipError_t lt_error(hipblasStatus_t s) {
    if (s == HIPBLAS_STATUS_SUCCESS)
        return hipSuccess;
    if (s == HIPBLAS_STATUS_ALLOC_FAILED)
        return hipErrorOutOfMemory;
    return hipErrorUnknown;
}

uint16_t bf16_bits_host(float x) {
    uint32_t u;
    std::memcpy(&u, &x, 4);
    if ((u & 0x7fffffffu) > 0x7f800000u)
        return (uint16_t)((u >> 16) | 0x40);   // quiet NaN
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// Elements per row of an activation buffer: rows start on 16-byte boundaries.
int row_ld(int n, int elem_bytes) {
    const int q = 16 / elem_bytes;
    return (n + q - 1) / q * q;
}

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

// ---- gather / scatter ------------------------------------------------------

// dst[r * ld + f] = feature f of sweep point b0 + r (bf16 bits or fp32);
// one thread per (point, feature), features fastest.
template <bool BF16>
__global__ void __launch_bounds__(256) layers_gather_kernel(DevMap m, int64_t b0, int64_t rows, int32_t ld,
                                                            void *__restrict__ dst) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int F = m.n_features;
    if (i >= rows * F)
        return;
    const int64_t r = i / F;
    const int f = (int)(i - r * F);
    int64_t p[HPACML_MAX_RANK];
    sweep_point(m, b0 + r, p);
    const float v = ldg(feature_ptr(m, p, interior(m, p), f));
    if (BF16)
        ((uint16_t *)dst)[r * ld + f] = (uint16_t)(__float_as_uint(round_bf16(v)) >> 16);
    else
        ((float *)dst)[r * ld + f] = v;
}

// Output g of sweep point b0 + r = src[r * ld + g].
__global__ void __launch_bounds__(256) layers_scatter_kernel(DevMap m, int64_t b0, int64_t rows, int32_t ld,
                                                             const float *__restrict__ src) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int G = m.n_features;
    if (i >= rows * G)
        return;
    const int64_t r = i / G;
    const int g = (int)(i - r * G);
    int64_t p[HPACML_MAX_RANK];
    sweep_point(m, b0 + r, p);
    stg(const_cast<float *>(feature_ptr(m, p, interior(m, p), g)), src[r * ld + g]);
}

typedef float float2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));

// Two floats to a packed pair of bf16 (nearest even, one conversion).
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
    const bf16x2v h = __builtin_convertvector((float2v){lo, hi}, bf16x2v);
    return __builtin_bit_cast(uint32_t, h);
}

// Gather + first layer: Y[r][n] = act(b[n] + sum_k W[n][k] x_r[k]) for the
// chunk's points r (x_r gathered through the map; bf16 models round x_r and
// Y to bf16, the weights are stored rounded).  KC = the input width rounded
// up to even; the weights come packed per neuron group ([group][V][KC]
// fp32, zero past the input width and past N) with the bias padded to the
// row width.  Thread t owns neuron group g = t % G (V consecutive neurons,
// weights in registers) for the points t / G, t / G + R, ... of each tile
// (R = 256 / G replicas); the row padding is written 0.
template <bool BF16, int KC>
__global__ void __launch_bounds__(256) layers_first_kernel(DevMap m, int64_t b0, int64_t rows,
                                                           const float *__restrict__ Wp,
                                                           const float *__restrict__ bias, int32_t G, int32_t relu,
                                                           int32_t ldy, void *__restrict__ Y) {
    constexpr int V = BF16 ? 8 : 4;   // neurons per thread: one 16-byte store per point
    __shared__ float2v xs[kTileP][KC / 2];
    const int F = m.n_features;
    const int R = 256 / G;
    const int t = threadIdx.x, g = t % G, rep = t / G;
    float w[V][KC], bb[V];
    {
        const float4 *src = (const float4 *)(Wp + (size_t)g * V * KC);
#pragma unroll
        for (int i = 0; i < V * KC / 4; ++i) {
            const float4 q = src[i];
            const float v4[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
            for (int e = 0; e < 4; ++e)
                w[(4 * i + e) / KC][(4 * i + e) % KC] = v4[e];
        }
        const float4 *bsrc = (const float4 *)(bias + g * V);
#pragma unroll
        for (int i = 0; i < V / 4; ++i) {
            const float4 q = bsrc[i];
            bb[4 * i] = q.x;
            bb[4 * i + 1] = q.y;
            bb[4 * i + 2] = q.z;
            bb[4 * i + 3] = q.w;
        }
    }
    const int64_t n_tiles = (rows + kTileP - 1) / kTileP;
    for (int64_t tile = blockIdx.x; tile < n_tiles; tile += gridDim.x) {
        const int64_t p0 = tile * kTileP;
        const int np = (int)(rows - p0 < kTileP ? rows - p0 : kTileP);
        __syncthreads();   // the previous tile's inputs are read
        float *xf = (float *)xs;
        for (int e = t; e < np * KC; e += 256) {
            const int pp = e / KC, f = e - pp * KC;
            float v = 0.f;
            if (f < F) {
                int64_t pt[HPACML_MAX_RANK];
                sweep_point(m, b0 + p0 + pp, pt);
                v = ldg(feature_ptr(m, pt, interior(m, pt), f));
                if (BF16)
                    v = round_bf16(v);
            }
            xf[e] = v;
        }
        __syncthreads();
        if (rep >= R)
            continue;
        for (int pp = rep; pp < np; pp += R) {
            float acc[V];
#pragma unroll
            for (int j = 0; j < V; ++j)
                acc[j] = bb[j];
#pragma unroll
            for (int k2 = 0; k2 < KC / 2; ++k2) {
                const float2v x2 = xs[pp][k2];
#pragma unroll
                for (int j = 0; j < V; ++j) {
                    acc[j] = fmaf(w[j][2 * k2], x2.x, acc[j]);
                    acc[j] = fmaf(w[j][2 * k2 + 1], x2.y, acc[j]);
                }
            }
            if (relu) {
#pragma unroll
                for (int j = 0; j < V; ++j)
                    acc[j] = relu_arith(acc[j]);
            }
            const int64_t row = p0 + pp;
            if (BF16) {
                uint4 o;
                o.x = pack_bf16(acc[0], acc[1]);
                o.y = pack_bf16(acc[2], acc[3]);
                o.z = pack_bf16(acc[4], acc[5]);
                o.w = pack_bf16(acc[6], acc[7]);
                *(uint4 *)((uint16_t *)Y + row * ldy + g * V) = o;
            } else {
                *(float4 *)((float *)Y + row * ldy + g * V) = make_float4(acc[0], acc[1], acc[2], acc[3]);
            }
        }
    }
}

// Last layer + scatter for FO <= 8 outputs and K <= 1024: output o of point r is
// act(b[o] + sum_k W[o][k] A[r][k]), written through the `from` map.  Eight
// lanes share a point and read its row in 128-byte segments (16 bytes per
// lane); the eight partial sums per output meet by xor shuffles, and lane
// o of the group writes output o.  Elements past K (row padding, which the
// matmuls leave unwritten) are skipped.
template <bool BF16, int FO>
__global__ void __launch_bounds__(256) layers_last_kernel(DevMap m, int64_t b0, int64_t rows, const void *A,
                                                          int32_t lda, int32_t K, const void *Wv, int32_t ldw,
                                                          const float *__restrict__ bias, int32_t relu) {
    constexpr int V = BF16 ? 8 : 4;   // elements per 16-byte load
    __shared__ float ws[FO][kLastMaxK];
    for (int e = threadIdx.x; e < FO * K; e += 256) {
        const int o = e / K, k = e - o * K;
        ws[o][k] = BF16 ? __uint_as_float((uint32_t)((const uint16_t *)Wv)[(size_t)o * ldw + k] << 16)
                        : ((const float *)Wv)[(size_t)o * ldw + k];
    }
    __syncthreads();
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int sub = lane & 7, q = lane >> 3;
    const int full = K / (8 * V);             // segments every lane of the group reads whole
    const bool tail = full * 8 * V < K;
    for (int64_t base = ((int64_t)blockIdx.x * 4 + wave) * 8; base < rows; base += (int64_t)gridDim.x * 32) {
        const int64_t r = base + q;
        const bool ok = r < rows;
        const int64_t rr = ok ? r : rows - 1;   // idle lanes read a valid row, results unused
        float acc[FO];
#pragma unroll
        for (int o = 0; o < FO; ++o)
            acc[o] = 0.f;
        auto segment = [&](int s, bool guard) {
            const int k0 = (s * 8 + sub) * V;
            if (guard && k0 >= K)
                return;
            float a[V];
            if (BF16) {
                const uint4 u = *(const uint4 *)((const uint16_t *)A + rr * lda + k0);
                const uint32_t h[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    a[2 * j] = __uint_as_float(h[j] << 16);
                    a[2 * j + 1] = __uint_as_float(h[j] & 0xffff0000u);
                }
            } else {
                const float4 u = *(const float4 *)((const float *)A + rr * lda + k0);
                a[0] = u.x;
                a[1] = u.y;
                a[2] = u.z;
                a[3] = u.w;
            }
#pragma unroll
            for (int j = 0; j < V; ++j) {
                if (!guard || k0 + j < K) {
#pragma unroll
                    for (int o = 0; o < FO; ++o)
                        acc[o] = fmaf(ws[o][k0 + j], a[j], acc[o]);
                }
            }
        };
        int s = 0;
        for (; s + 4 <= full; s += 4) {
#pragma unroll
            for (int u = 0; u < 4; ++u)
                segment(s + u, false);
        }
        for (; s < full; ++s)
            segment(s, false);
        if (tail)
            segment(full, true);
        float y = 0.f;
#pragma unroll
        for (int o = 0; o < FO; ++o) {
            float v = acc[o];
            v += __shfl_xor(v, 1);
            v += __shfl_xor(v, 2);
            v += __shfl_xor(v, 4);
            if (o == sub)
                y = v;
        }
        if (ok && sub < FO) {
            y += bias[sub];
            if (relu)
                y = relu_arith(y);
            int64_t pt[HPACML_MAX_RANK];
            sweep_point(m, b0 + r, pt);
            stg(const_cast<float *>(feature_ptr(m, pt, interior(m, pt), sub)), y);
        }
    }
}

}  // namespace

// ---- the plan ----------------------------------------------------------------

struct LayersPlan {
    int n_layers = 0, device = 0;
    bool bf16 = false;
    std::vector<int> K, N, ld_in, ld_out, act;
    void *wbuf = nullptr;                // weights ([N][ld_in] per layer), then fp32 biases
    std::vector<const void *> W;
    std::vector<const float *> bias;
    int64_t chunk = 0;                   // points per chunk
    bool first_fused = false;            // first layer in the gather kernel
    bool last_fused = false;             // last layer in the scatter kernel
    int g0 = 0, g1 = 0;                  // layers [g0, g1) are matmuls
    const float *first_w = nullptr;      // first layer packed per neuron group ([G][V][KC] fp32)
    const float *first_b = nullptr;      // its bias, zero-padded to G * V
    int first_kc = 0, first_g = 0;
    hipblasLtHandle_t lt = nullptr;
    std::vector<hipblasLtMatmulDesc_t> op;
    std::vector<hipblasLtMatrixLayout_t> la;
    bool desc_ok = false;
    struct Cols {                        // per chunk size: layouts of X and D, algorithms (matmul layers)
        bool ok = false;
        std::vector<hipblasLtMatrixLayout_t> lb, ld;
        std::vector<hipblasLtMatmulAlgo_t> algo;
        size_t ws_need = 0;
    };
    std::map<int64_t, Cols> cols;
    std::mutex mu;
    void *ws = nullptr;                  // [act A][act B][fp32 output rows][library scratch]
    size_t ws_bytes = 0;
};

namespace {

hipDataType act_type(const LayersPlan &p) { return p.bf16 ? HIP_R_16BF : HIP_R_32F; }
int act_bytes(const LayersPlan &p) { return p.bf16 ? 2 : 4; }

// Element count of the larger activation buffer per point.
int64_t buf_ld(const LayersPlan &p) {
    int64_t m = p.ld_in[0];
    for (int l = 0; l + 1 < p.n_layers; ++l)
        m = std::max<int64_t>(m, p.ld_out[l]);
    return m;
}

void drop_descs(LayersPlan &p) {
    for (auto x : p.la)
        (void)hipblasLtMatrixLayoutDestroy(x);
    for (auto x : p.op)
        (void)hipblasLtMatmulDescDestroy(x);
    p.la.clear();
    p.op.clear();
}

bool make_descs_once(LayersPlan &p) {
    p.lt = lt_handle(p.device);
    if (!p.lt)
        return false;
    const hipDataType dt = act_type(p);
    for (int l = 0; l < p.n_layers; ++l) {
        hipblasLtMatmulDesc_t d = nullptr;
        if (hipblasLtMatmulDescCreate(&d, HIPBLAS_COMPUTE_32F, HIP_R_32F) != HIPBLAS_STATUS_SUCCESS)
            return false;
        p.op.push_back(d);
        const int32_t ta = HIPBLAS_OP_T, tb = HIPBLAS_OP_N;
        const uint32_t epi = p.act[l] == HPACML_ACT_RELU ? HIPBLASLT_EPILOGUE_RELU_BIAS : HIPBLASLT_EPILOGUE_BIAS;
        const void *bp = p.bias[l];
        const int32_t bt = HIP_R_32F;
        if (hipblasLtMatmulDescSetAttribute(d, HIPBLASLT_MATMUL_DESC_TRANSA, &ta, sizeof ta) ||
            hipblasLtMatmulDescSetAttribute(d, HIPBLASLT_MATMUL_DESC_TRANSB, &tb, sizeof tb) ||
            hipblasLtMatmulDescSetAttribute(d, HIPBLASLT_MATMUL_DESC_EPILOGUE, &epi, sizeof epi) ||
            hipblasLtMatmulDescSetAttribute(d, HIPBLASLT_MATMUL_DESC_BIAS_POINTER, &bp, sizeof bp) ||
            hipblasLtMatmulDescSetAttribute(d, HIPBLASLT_MATMUL_DESC_BIAS_DATA_TYPE, &bt, sizeof bt))
            return false;
        // stored weights: column-major K x N (row n of W is column n), read transposed
        hipblasLtMatrixLayout_t a = nullptr;
        if (hipblasLtMatrixLayoutCreate(&a, dt, p.K[l], p.N[l], p.ld_in[l]) != HIPBLAS_STATUS_SUCCESS)
            return false;
        p.la.push_back(a);
    }
    return true;
}

// Matmul descriptors and weight layouts of every layer (made once).
bool make_descs(LayersPlan &p) {
    if (p.desc_ok)
        return true;
    p.desc_ok = make_descs_once(p);
    if (!p.desc_ok)
        drop_descs(p);
    return p.desc_ok;
}

void drop_cols(LayersPlan::Cols &e) {
    for (auto x : e.lb)
        if (x)
            (void)hipblasLtMatrixLayoutDestroy(x);
    for (auto x : e.ld)
        if (x)
            (void)hipblasLtMatrixLayoutDestroy(x);
    e.lb.clear();
    e.ld.clear();
}

// Layouts and algorithms for chunks of c points (cached).
LayersPlan::Cols *cols_for(LayersPlan &p, int64_t c) {
    auto it = p.cols.find(c);
    if (it != p.cols.end())
        return it->second.ok ? &it->second : nullptr;
    if (p.cols.size() >= 16) {
        // a bounded cache: forget every size but the full chunk (which a
        // caller may hold while it asks for its tail)
        for (auto kv = p.cols.begin(); kv != p.cols.end();) {
            if (kv->first == p.chunk) {
                ++kv;
                continue;
            }
            drop_cols(kv->second);
            kv = p.cols.erase(kv);
        }
    }
    LayersPlan::Cols &e = p.cols[c];
    e.lb.assign(p.n_layers, nullptr);
    e.ld.assign(p.n_layers, nullptr);
    e.algo.assign(p.n_layers, hipblasLtMatmulAlgo_t{});
    if (p.g0 == p.g1) {      // no matmul layer
        e.ok = true;
        return &e;
    }
    if (!make_descs(p))
        return nullptr;
    hipblasLtMatmulPreference_t pref = nullptr;
    if (hipblasLtMatmulPreferenceCreate(&pref) != HIPBLAS_STATUS_SUCCESS)
        return nullptr;
    const uint64_t wsmax = kLibWorkspace;
    (void)hipblasLtMatmulPreferenceSetAttribute(pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &wsmax,
                                                sizeof wsmax);
    bool ok = true;
    for (int l = p.g0; l < p.g1 && ok; ++l) {
        const bool last = l + 1 == p.n_layers;
        ok = hipblasLtMatrixLayoutCreate(&e.lb[l], act_type(p), p.K[l], c, p.ld_in[l]) == HIPBLAS_STATUS_SUCCESS &&
             hipblasLtMatrixLayoutCreate(&e.ld[l], last ? HIP_R_32F : act_type(p), p.N[l], c, p.ld_out[l]) ==
                 HIPBLAS_STATUS_SUCCESS;
        if (!ok)
            break;
        // the library's ranking, first candidate whose scratch fits (the
        // preference alone does not always bound it)
        hipblasLtMatmulHeuristicResult_t res[kCandidates];
        int n = 0;
        ok = hipblasLtMatmulAlgoGetHeuristic(p.lt, p.op[l], p.la[l], e.lb[l], e.ld[l], e.ld[l], pref, kCandidates,
                                             res, &n) == HIPBLAS_STATUS_SUCCESS;
        int pick = -1;
        for (int i = 0; ok && i < n && pick < 0; ++i)
            if (res[i].state == HIPBLAS_STATUS_SUCCESS && res[i].workspaceSize <= kLibWorkspace)
                pick = i;
        ok = ok && pick >= 0;
        if (ok) {
            e.algo[l] = res[pick].algo;
            e.ws_need = std::max(e.ws_need, res[pick].workspaceSize);
        }
    }
    (void)hipblasLtMatmulPreferenceDestroy(pref);
    e.ok = ok;
    return ok ? &e : nullptr;
}

}  // namespace

namespace {

template <bool BF16>
void launch_first(const LayersPlan &p, const DevMap &in, int64_t b0, int64_t c, void *y, hipStream_t st) {
    const int64_t blocks = std::min<int64_t>((c + kTileP - 1) / kTileP, 1024);
    const int32_t relu = p.act[0] == HPACML_ACT_RELU;
#define HPACML_FIRST(KC)                                                                                    \
    case KC:                                                                                                \
        hipLaunchKernelGGL((layers_first_kernel<BF16, KC>), dim3((unsigned)blocks), dim3(256), 0, st, in, b0, c, \
                           p.first_w, p.first_b, p.first_g, relu, p.ld_out[0], y);                           \
        break;
    switch (p.first_kc) {
        HPACML_FIRST(2)
        HPACML_FIRST(4)
        HPACML_FIRST(6)
        HPACML_FIRST(8)
        HPACML_FIRST(10)
        HPACML_FIRST(12)
    }
#undef HPACML_FIRST
}

template <bool BF16>
void launch_last(const LayersPlan &p, const DevMap &out, int64_t b0, int64_t c, const void *x, hipStream_t st) {
    const int L = p.n_layers;
    const int64_t blocks = std::min<int64_t>((c + 31) / 32, 1024);
    const int32_t relu = p.act[L - 1] == HPACML_ACT_RELU;
#define HPACML_LAST(FO)                                                                                      \
    case FO:                                                                                                 \
        hipLaunchKernelGGL((layers_last_kernel<BF16, FO>), dim3((unsigned)blocks), dim3(256), 0, st, out, b0, c, x, \
                           p.ld_in[L - 1], p.K[L - 1], p.W[L - 1], p.ld_in[L - 1], p.bias[L - 1], relu);      \
        break;
    switch (p.N[L - 1]) {
        HPACML_LAST(1)
        HPACML_LAST(2)
        HPACML_LAST(3)
        HPACML_LAST(4)
        HPACML_LAST(5)
        HPACML_LAST(6)
        HPACML_LAST(7)
        HPACML_LAST(8)
    }
#undef HPACML_LAST
}

}  // namespace

hipError_t layers_create(int n_layers, const int32_t *dims, const int32_t *act, const float *const *W,
                         const float *const *b, int compute, LayersPlan **out) {
    *out = nullptr;
    LayersPlan *p = new LayersPlan();
    hipError_t e = hipGetDevice(&p->device);
    if (e != hipSuccess) {
        delete p;
        return e;
    }
    p->n_layers = n_layers;
    p->bf16 = compute == HPACML_BF16;
    const int eb = p->bf16 ? 2 : 4;
    size_t bytes = 0;
    std::vector<size_t> woff(n_layers), boff(n_layers);
    for (int l = 0; l < n_layers; ++l) {
        p->K.push_back(dims[l]);
        p->N.push_back(dims[l + 1]);
        p->ld_in.push_back(row_ld(dims[l], eb));
        p->ld_out.push_back(row_ld(dims[l + 1], l + 1 == n_layers ? 4 : eb));
        p->act.push_back(act[l]);
        woff[l] = bytes;
        bytes = align256(bytes + (size_t)p->N[l] * p->ld_in[l] * eb);
    }
    for (int l = 0; l < n_layers; ++l) {
        boff[l] = bytes;
        bytes = align256(bytes + (size_t)p->N[l] * 4);
    }
    // the first-layer kernel gives each of its 256 threads one group of V1
    // neurons: at most 2048 (bf16) or 1024 (fp32) neurons
    const int V1 = p->bf16 ? 8 : 4, KC = (dims[0] + 1) / 2 * 2;
    const int G1 = (dims[1] + V1 - 1) / V1;
    const bool first_fused = n_layers >= 2 && dims[0] <= kFirstMaxK && G1 <= 256;
    size_t fw_off = 0, fb_off = 0;
    if (first_fused) {
        fw_off = bytes;
        bytes = align256(bytes + (size_t)G1 * V1 * KC * 4);
        fb_off = bytes;
        bytes = align256(bytes + (size_t)G1 * V1 * 4);
    }
    std::vector<uint8_t> host(bytes, 0);
    if (first_fused) {
        // zero past the input width and past N (the buffer starts zeroed)
        float *fw = (float *)&host[fw_off];
        float *fb = (float *)&host[fb_off];
        for (int n = 0; n < dims[1]; ++n) {
            for (int k = 0; k < dims[0]; ++k) {
                const float v = W[0][(size_t)n * dims[0] + k];
                float r = v;
                if (p->bf16) {
                    const uint32_t u = (uint32_t)bf16_bits_host(v) << 16;
                    std::memcpy(&r, &u, 4);
                }
                fw[(size_t)n * KC + k] = r;   // [g][j][k] with n = g * V + j
            }
            fb[n] = b[0][n];
        }
    }
    for (int l = 0; l < n_layers; ++l) {
        for (int o = 0; o < p->N[l]; ++o)
            for (int k = 0; k < p->K[l]; ++k) {
                const float w = W[l][(size_t)o * p->K[l] + k];
                const size_t at = woff[l] + ((size_t)o * p->ld_in[l] + k) * eb;
                if (p->bf16) {
                    const uint16_t h = bf16_bits_host(w);
                    std::memcpy(&host[at], &h, 2);
                } else {
                    std::memcpy(&host[at], &w, 4);
                }
            }
        std::memcpy(&host[boff[l]], b[l], (size_t)p->N[l] * 4);
    }
    e = hipMalloc(&p->wbuf, bytes);
    if (e == hipSuccess)
        e = hipMemcpy(p->wbuf, host.data(), bytes, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        layers_destroy(p);
        return e;
    }
    for (int l = 0; l < n_layers; ++l) {
        p->W.push_back((const uint8_t *)p->wbuf + woff[l]);
        p->bias.push_back((const float *)((const uint8_t *)p->wbuf + boff[l]));
    }
    if (first_fused) {
        p->first_w = (const float *)((const uint8_t *)p->wbuf + fw_off);
        p->first_b = (const float *)((const uint8_t *)p->wbuf + fb_off);
        p->first_kc = KC;
        p->first_g = G1;
    }
    // points per chunk: one activation buffer of about 1 GB (fewer, larger
    // matmuls; measured faster than chunks that fit the 256 MB last-level
    // cache); the environment variable HPACML_LAYERS_CHUNK_MB sets another size
    // (1 MB to 64 GB; other values are ignored), which also bounds the gather
    // and scatter grids (chunk x features < 2^31 x 256 threads)
    size_t target = (size_t)1024 << 20;
    if (const char *s = std::getenv("HPACML_LAYERS_CHUNK_MB")) {
        const long v = std::atol(s);
        if (v > 0 && v <= (1L << 16))
            target = (size_t)v << 20;
    }
    p->first_fused = first_fused;
    p->last_fused = n_layers >= 2 && dims[n_layers] <= kLastMaxOut && dims[n_layers - 1] <= kLastMaxK;
    p->g0 = p->first_fused ? 1 : 0;
    p->g1 = p->last_fused ? n_layers - 1 : n_layers;
    const int64_t per = buf_ld(*p) * eb;
    p->chunk = std::max<int64_t>(4096, (int64_t)(target / (size_t)per) / 256 * 256);
    *out = p;
    return hipSuccess;
}

void layers_destroy(LayersPlan *p) {
    if (!p)
        return;
    for (auto &kv : p->cols)
        drop_cols(kv.second);
    drop_descs(*p);
    (void)hipFree(p->wbuf);
    (void)hipFree(p->ws);
    delete p;
}

bool layers_ready(LayersPlan *p, int64_t n_points) {
    if (!p)
        return false;
    if (n_points <= 0)
        return true;
    std::lock_guard<std::mutex> lock(p->mu);
    const int64_t c = std::min(n_points, p->chunk), tail = n_points % p->chunk;
    if (!cols_for(*p, c))
        return false;
    return n_points <= p->chunk || tail == 0 || cols_for(*p, tail) != nullptr;
}

const char *layers_name(const LayersPlan *p) { return p->bf16 ? "mlp_layers_bf16" : "mlp_layers_f32"; }

hipError_t layers_infer(LayersPlan *p, const DevMap &in, const DevMap &out, hipStream_t stream) {
    const int64_t B = in.n_points;
    if (B == 0)
        return hipSuccess;
    std::lock_guard<std::mutex> lock(p->mu);
    const int64_t chunk = std::min(B, p->chunk);
    LayersPlan::Cols *full = cols_for(*p, chunk);
    const int64_t tail = B % chunk;
    LayersPlan::Cols *part = tail ? cols_for(*p, tail) : full;
    if (!full || !part)
        return hipErrorNotSupported;
    const int eb = act_bytes(*p);
    const int L = p->n_layers;
    const size_t act_b = align256((size_t)chunk * buf_ld(*p) * eb);
    const size_t out_b = p->last_fused ? 0 : align256((size_t)chunk * p->ld_out[L - 1] * 4);
    const size_t lib_b = std::max(full->ws_need, part->ws_need);
    const size_t need = 2 * act_b + out_b + lib_b;
    if (p->ws_bytes < need) {
        void *buf = nullptr;
        hipError_t e = hipMalloc(&buf, need);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            return e;
        }
        // the old workspace may still be in use by work queued on this stream
        e = hipStreamSynchronize(stream);
        (void)hipFree(p->ws);
        p->ws = buf;
        p->ws_bytes = need;
        if (e != hipSuccess)
            return e;
    }
    uint8_t *bufA = (uint8_t *)p->ws, *bufB = bufA + act_b;
    float *ybuf = (float *)(bufB + act_b);
    void *lib = lib_b ? (void *)(bufB + act_b + out_b) : nullptr;
    const float one = 1.f, zero = 0.f;
    for (int64_t b0 = 0; b0 < B; b0 += chunk) {
        const int64_t c = std::min(chunk, B - b0);
        LayersPlan::Cols *cc = c == chunk ? full : part;
        // the input of layer g0 into bufA
        if (p->first_fused) {
            if (p->bf16)
                launch_first<true>(*p, in, b0, c, bufA, stream);
            else
                launch_first<false>(*p, in, b0, c, bufA, stream);
        } else {
            const int64_t blocks = (c * in.n_features + 255) / 256;
            if (p->bf16)
                hipLaunchKernelGGL(layers_gather_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, stream, in, b0,
                                   c, p->ld_in[0], (void *)bufA);
            else
                hipLaunchKernelGGL(layers_gather_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, stream, in,
                                   b0, c, p->ld_in[0], (void *)bufA);
        }
        hipError_t e = hipGetLastError();
        if (e != hipSuccess)
            return e;
        uint8_t *x = bufA, *y = bufB;
        for (int l = p->g0; l < p->g1; ++l) {
            void *d = l + 1 == L ? (void *)ybuf : (void *)y;
            e = lt_error(hipblasLtMatmul(p->lt, p->op[l], &one, p->W[l], p->la[l], x, cc->lb[l], &zero, d,
                                         cc->ld[l], d, cc->ld[l], &cc->algo[l], lib, lib_b, stream));
            if (e != hipSuccess)
                return e;
            std::swap(x, y);
        }
        if (p->last_fused) {
            // x holds the input rows of the last layer
            if (p->bf16)
                launch_last<true>(*p, out, b0, c, x, stream);
            else
                launch_last<false>(*p, out, b0, c, x, stream);
        } else {
            const int64_t blocks = (c * out.n_features + 255) / 256;
            hipLaunchKernelGGL(layers_scatter_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, out, b0, c,
                               p->ld_out[L - 1], (const float *)ybuf);
        }
        e = hipGetLastError();
        if (e != hipSuccess)
            return e;
    }
    return hipSuccess;
}

}  // namespace hpacml
