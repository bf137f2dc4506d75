// Layer-by-layer MLP inference (Sec. IV-B: the surrogate is a stack of
// Linear/ReLU layers evaluated on the gathered input tensor) for shapes the
// fused kernels do not take: widths above 512 (bf16) or 128 (fp32), more
// hidden layers, non-uniform stacks, and maps outside the 32-bit form.
//
// A chunk of points goes through: a gather kernel (the map's input tensor as
// rows of bf16 or fp32), one hipBLASLt matmul per layer, and a scatter
// kernel (fp32 output rows through the `from` map).  Each matmul computes,
// column-major, D[N x C] = W[N x K] X[K x C] with the layer's bias and ReLU
// applied to the fp32 accumulators in its epilogue; hidden activations of a
// bf16 model are stored as bf16 (nearest-even), the last layer's output as
// fp32 -- the rounding points of the fused kernels.  Chunks are sized so one
// activation buffer stays near the 256 MB last-level cache.
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
    hipblasLtHandle_t lt = nullptr;
    std::vector<hipblasLtMatmulDesc_t> op;
    std::vector<hipblasLtMatrixLayout_t> la;
    bool desc_ok = false;
    struct Cols {                        // per chunk size: layouts of X and D, algorithms
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
            for (auto x : kv->second.lb)
                (void)hipblasLtMatrixLayoutDestroy(x);
            for (auto x : kv->second.ld)
                (void)hipblasLtMatrixLayoutDestroy(x);
            kv = p.cols.erase(kv);
        }
    }
    LayersPlan::Cols &e = p.cols[c];
    if (!make_descs(p))
        return nullptr;
    hipblasLtMatmulPreference_t pref = nullptr;
    if (hipblasLtMatmulPreferenceCreate(&pref) != HIPBLAS_STATUS_SUCCESS)
        return nullptr;
    const uint64_t wsmax = kLibWorkspace;
    (void)hipblasLtMatmulPreferenceSetAttribute(pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &wsmax,
                                                sizeof wsmax);
    bool ok = true;
    for (int l = 0; l < p.n_layers && ok; ++l) {
        const bool last = l + 1 == p.n_layers;
        hipblasLtMatrixLayout_t b = nullptr, d = nullptr;
        ok = hipblasLtMatrixLayoutCreate(&b, act_type(p), p.K[l], c, p.ld_in[l]) == HIPBLAS_STATUS_SUCCESS &&
             hipblasLtMatrixLayoutCreate(&d, last ? HIP_R_32F : act_type(p), p.N[l], c, p.ld_out[l]) ==
                 HIPBLAS_STATUS_SUCCESS;
        if (b)
            e.lb.push_back(b);
        if (d)
            e.ld.push_back(d);
        if (!ok)
            break;
        // the library's ranking, first candidate whose scratch fits (the
        // preference alone does not always bound it)
        hipblasLtMatmulHeuristicResult_t res[kCandidates];
        int n = 0;
        ok = hipblasLtMatmulAlgoGetHeuristic(p.lt, p.op[l], p.la[l], b, d, d, pref, kCandidates, res, &n) ==
             HIPBLAS_STATUS_SUCCESS;
        int pick = -1;
        for (int i = 0; ok && i < n && pick < 0; ++i)
            if (res[i].state == HIPBLAS_STATUS_SUCCESS && res[i].workspaceSize <= kLibWorkspace)
                pick = i;
        ok = ok && pick >= 0;
        if (ok) {
            e.algo.push_back(res[pick].algo);
            e.ws_need = std::max(e.ws_need, res[pick].workspaceSize);
        }
    }
    (void)hipblasLtMatmulPreferenceDestroy(pref);
    e.ok = ok;
    return ok ? &e : nullptr;
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
    std::vector<uint8_t> host(bytes, 0);
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
    // points per chunk: one activation buffer of about 256 MB (the
    // environment variable HPACML_LAYERS_CHUNK_MB overrides the size)
    size_t target = (size_t)256 << 20;
    if (const char *s = std::getenv("HPACML_LAYERS_CHUNK_MB")) {
        const long v = std::atol(s);
        if (v > 0 && v <= (1L << 20))
            target = (size_t)v << 20;
    }
    const int64_t per = buf_ld(*p) * eb;
    p->chunk = std::max<int64_t>(4096, (int64_t)(target / (size_t)per) / 256 * 256);
    *out = p;
    return hipSuccess;
}

void layers_destroy(LayersPlan *p) {
    if (!p)
        return;
    for (auto &kv : p->cols) {
        for (auto x : kv.second.lb)
            (void)hipblasLtMatrixLayoutDestroy(x);
        for (auto x : kv.second.ld)
            (void)hipblasLtMatrixLayoutDestroy(x);
    }
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
    const size_t act_b = align256((size_t)chunk * buf_ld(*p) * eb);
    const size_t out_b = align256((size_t)chunk * p->ld_out[p->n_layers - 1] * 4);
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
        int64_t blocks = (c * in.n_features + 255) / 256;
        if (p->bf16)
            hipLaunchKernelGGL(layers_gather_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, stream, in, b0, c,
                               p->ld_in[0], (void *)bufA);
        else
            hipLaunchKernelGGL(layers_gather_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, stream, in, b0,
                               c, p->ld_in[0], (void *)bufA);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess)
            return e;
        uint8_t *x = bufA, *y = bufB;
        for (int l = 0; l < p->n_layers; ++l) {
            void *d = l + 1 == p->n_layers ? (void *)ybuf : (void *)y;
            e = lt_error(hipblasLtMatmul(p->lt, p->op[l], &one, p->W[l], p->la[l], x, cc->lb[l], &zero, d,
                                         cc->ld[l], d, cc->ld[l], &cc->algo[l], lib, lib_b, stream));
            if (e != hipSuccess)
                return e;
            std::swap(x, y);
        }
        blocks = (c * out.n_features + 255) / 256;
        hipLaunchKernelGGL(layers_scatter_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, out, b0, c,
                           p->ld_out[p->n_layers - 1], (const float *)ybuf);
        e = hipGetLastError();
        if (e != hipSuccess)
            return e;
    }
    return hipSuccess;
}

}  // namespace hpacml
