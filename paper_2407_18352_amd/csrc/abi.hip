// C ABI of the library: handle management, validation and kernel dispatch.
// Declarations and the contract of every entry point are in include/hpacml.h.
#include <hip/hip_runtime.h>

#include <cstring>
#include <mutex>
#include <set>
#include <string>
#include <new>
#include <vector>

#include "hpacml.h"
#include "cnn.hpp"
#include "kernels.hpp"
#include "layers.hpp"
#include "plan.hpp"

using namespace hpacml;

struct hpacml_map_s {
    MapPlan plan;
    int device = 0;
    FeatureEntry *feat_dev = nullptr;
    float **base_dev = nullptr;
    int64_t *stride_dev = nullptr;
    DevMap dev{};
    Map32 m32{};
    bool fast = false;   // m32 is valid
    bool t32 = false;    // tab is valid: 32-bit view, raw8, at most 64 features
    FeatTable32 tab{};
    FeatTable32 *tab_dev = nullptr;   // device copy of tab (kernels that index it per thread)
    // snapshot of this (TO) map's inputs for inferences whose outputs may
    // overwrite them: a [points x features] record and a map over it,
    // created on first use
    mutable std::mutex snap_mu;
    mutable float *snap = nullptr;
    mutable hpacml_map *snap_map = nullptr;
};

enum class Variant { Generic, F32, BF16, BF16R };

struct hpacml_model_s {
    int32_t n_layers = 0, compute = 0;
    std::vector<int32_t> dims, act;
    int device = 0;
    Variant variant = Variant::Generic;
    float *gen_buf = nullptr;   // generic-kernel weights and biases
    DevModel gen{};
    float *f32_img = nullptr;   // packed LDS image of the fp32 kernel
    F32Packed f32{};
    uint16_t *bf16_frags = nullptr;  // packed fragments of the bf16 kernel
    BF16Packed bf16{};
    uint8_t *bf16r_buf = nullptr;    // weight stream, output fragments, biases of the register-resident bf16 kernel
    BF16RPacked bf16r{};
    bool padded = false;             // the fast kernel runs the hidden layers zero-padded to its width
    LayersPlan *layers = nullptr;    // layer-by-layer path (matmul library), in place of the general kernel
    std::string fast_name;           // its name (with "_padded" then)
    // convolutional models
    bool cnn = false;
    CnnPlan cnnp;
    float *cnn_buf = nullptr;        // the caller's layouts, every layer
    std::vector<CnnLayerDev> cnn_layers;
    bool cnn_fused = false;          // the fused kernel takes this stack
    float *fused_buf = nullptr;      // its packed weights
    CnnFused fused{};
    std::mutex ws_mu;                // layer-by-layer workspace, grown on demand
    float *ws = nullptr;
    int64_t ws_floats = 0;
};

namespace {

hpacml_status hip_status(hipError_t e) {
    if (e == hipSuccess)
        return HPACML_OK;
    if (e == hipErrorOutOfMemory)
        return HPACML_E_NOMEM;
    return HPACML_E_DEVICE;
}

// Round to bf16 (nearest even; NaN stays a quiet NaN) and back to fp32.
float host_bf16(float x) {
    uint32_t u;
    std::memcpy(&u, &x, 4);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) {
        u = (u | 0x00400000u) & 0xFFFF0000u;
    } else {
        u += 0x7FFFu + ((u >> 16) & 1u);
        u &= 0xFFFF0000u;
    }
    float r;
    std::memcpy(&r, &u, 4);
    return r;
}

// Every target must be device memory of the current device, and the elements
// the map can address must lie inside that allocation.
hpacml_status check_device_targets(const MapPlan &p, int device) {
    for (int t = 0; t < p.n_targets; ++t) {
        hipPointerAttribute_t attr;
        if (hipPointerGetAttributes(&attr, p.base[t]) != hipSuccess) {
            (void)hipGetLastError();
            return HPACML_E_INVAL;
        }
        if (attr.type != hipMemoryTypeDevice && attr.type != hipMemoryTypeManaged)
            return HPACML_E_INVAL;
        if (attr.device != device)
            return HPACML_E_INVAL;
        hipDeviceptr_t abase = nullptr;
        size_t asize = 0;
        if (hipMemGetAddressRange(&abase, &asize, (hipDeviceptr_t)p.base[t]) != hipSuccess) {
            (void)hipGetLastError();
            return HPACML_E_INVAL;
        }
        const char *lo = (const char *)abase, *hi = lo + asize;
        const char *a = (const char *)p.base[t];
        if (a < lo || a + 4 * (p.max_elem[t] + 1) > hi)
            return HPACML_E_RANGE;
        if (((uintptr_t)a & 3u) != 0)
            return HPACML_E_INVAL;
    }
    return HPACML_OK;
}

template <typename T>
hpacml_status upload(T **dst, const T *src, size_t n) {
    *dst = nullptr;
    if (n == 0)
        return HPACML_OK;
    hipError_t e = hipMalloc((void **)dst, n * sizeof(T));
    if (e != hipSuccess) {
        *dst = nullptr;
        return hip_status(e);
    }
    e = hipMemcpy(*dst, src, n * sizeof(T), hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        (void)hipFree(*dst);
        *dst = nullptr;
        return hip_status(e);
    }
    return HPACML_OK;
}

bool same_device(int dev) {
    int cur = -1;
    return hipGetDevice(&cur) == hipSuccess && cur == dev;
}

hpacml_status check_infer(const hpacml_model *model, const hpacml_map *in, const hpacml_map *out,
                          bool *snapshot = nullptr) {
    if (!model || !in || !out)
        return HPACML_E_INVAL;
    if (in->plan.dir != HPACML_TO || out->plan.dir != HPACML_FROM)
        return HPACML_E_INVAL;
    if (model->cnn) {
        // images: the last two sweep dimensions; leading ones number the images
        const CnnPlan &c = model->cnnp;
        const MapPlan &ip = in->plan;
        if (ip.rank < 2 || ip.count[ip.rank - 2] != c.height || ip.count[ip.rank - 1] != c.width ||
            ip.n_features != c.in_channels)
            return HPACML_E_SHAPE;
        const int64_t S = ip.n_points / ((int64_t)c.height * c.width);
        const CnnShape &o = c.shape[c.n_layers];
        if (out->plan.n_points != S * o.h * o.w || out->plan.n_features != o.c)
            return HPACML_E_SHAPE;
    } else {
        if (in->plan.n_points != out->plan.n_points)
            return HPACML_E_SHAPE;
        if (in->plan.n_features != model->dims[0] || out->plan.n_features != model->dims[model->n_layers])
            return HPACML_E_SHAPE;
    }
    if (in->device != model->device || out->device != model->device || !same_device(model->device))
        return HPACML_E_INVAL;
    const Overlap ov = classify_overlap(in->plan, out->plan);
    if (ov == Overlap::OutputRace)
        return HPACML_E_ALIAS;
    if (snapshot)
        *snapshot = ov == Overlap::Snapshot;
    return HPACML_OK;
}

}  // namespace

hpacml_status hpacml::infer_status(const hpacml_model *model, const hpacml_map *in, const hpacml_map *out) {
    return check_infer(model, in, out);
}

namespace hpacml {

DevMap make_devmap(const MapPlan &p, const FeatureEntry *feat_dev, float *const *base_dev,
                   const int64_t *stride_dev) {
    DevMap m{};
    m.rank = p.rank;
    m.n_features = p.n_features;
    m.n_targets = p.n_targets;
    m.pointwise = p.pointwise ? 1 : 0;
    m.n_points = p.n_points;
    bool small = p.n_points < (int64_t(1) << 31);
    for (int d = 0; d < HPACML_MAX_RANK; ++d) {
        m.count[d] = p.count[d];
        m.start[d] = p.start[d];
        m.step[d] = p.step[d];
        m.extent[d] = p.extent[d];
        m.bnd[d] = p.bnd[d];
        m.omin[d] = p.omin[d];
        m.omax[d] = p.omax[d];
        m.stride0[d] = d < p.rank ? p.stride[d] : 0;
        small = small && p.count[d] < (int64_t(1) << 31) && p.count[d] > 0;
    }
    m.small_counts = small ? 1 : 0;
    m.same_strides = 1;
    for (int t = 1; t < p.n_targets; ++t)
        for (int d = 0; d < p.rank; ++d)
            if (p.stride[(size_t)t * 4 + d] != p.stride[d])
                m.same_strides = 0;
    m.feat = feat_dev;
    m.base = base_dev;
    m.stride = stride_dev;
    return m;
}

// Division by m->count[d]: n / c == (n * magic) >> (31 + l) for n < 2^31,
// l = ceil(log2 c); false when the multiplier does not fit or a probe fails.
bool set_div_magic(Map32 *m, int d) {
    const uint64_t dv = (uint64_t)m->count[d];
    int l = 0;
    while ((uint64_t(1) << l) < dv)
        ++l;
    const uint64_t magic = ((uint64_t(1) << (31 + l)) + dv - 1) / dv;
    if (magic > UINT32_MAX)
        return false;
    m->magic[d] = (uint32_t)magic;
    m->shift[d] = 31 + l;
    const uint32_t probes[6] = {0u, (uint32_t)dv - 1u, (uint32_t)dv, (uint32_t)(2 * dv - 1), (uint32_t)INT32_MAX,
                                (uint32_t)INT32_MAX - 1u};
    for (uint32_t n : probes)
        if ((uint32_t)(((uint64_t)n * m->magic[d]) >> m->shift[d]) != n / (uint32_t)dv)
            return false;
    return true;
}

bool make_map32(const MapPlan &p, Map32 *out) {
    const int64_t lim = INT32_MAX;
    Map32 m{};
    if (p.n_points >= lim || !p.idx32)
        return false;
    for (int t = 1; t < p.n_targets; ++t)
        for (int d = 0; d < p.rank; ++d)
            if (p.stride[(size_t)t * 4 + d] != p.stride[d])
                return false;
    for (const FeatureEntry &e : p.feat)
        if (e.delta > lim || e.delta < -lim)
            return false;
    m.rank = p.rank;
    m.n_features = p.n_features;
    m.n_targets = p.n_targets;
    m.n_points = (int32_t)p.n_points;
    for (int d = 0; d < HPACML_MAX_RANK; ++d) {
        const bool used = d < p.rank;
        if (used && (p.count[d] < 1 || p.start[d] + p.count[d] * p.step[d] > 2 * lim / 3 ||
                     p.extent[d] > lim / 3 || p.stride[d] > lim || p.omin[d] < -lim / 3 || p.omax[d] > lim / 3))
            return false;
        m.count[d] = used ? (int32_t)p.count[d] : 1;
        m.start[d] = used ? (int32_t)p.start[d] : 0;
        m.step[d] = used ? (int32_t)p.step[d] : 1;
        m.extent[d] = used ? (int32_t)p.extent[d] : 1;
        m.stride[d] = used ? (int32_t)p.stride[d] : 0;
        m.bnd[d] = p.bnd[d];
        m.omin[d] = p.omin[d];
        m.omax[d] = p.omax[d];
        if (!set_div_magic(&m, d))
            return false;
    }
    *out = m;
    return true;
}

bool table32_supported(const MapPlan &p, bool map32) {
    return map32 && p.raw8 && p.n_features >= 1 && p.n_features <= kTableMaxF;
}

void table32_make(const MapPlan &p, FeatTable32 *out) {
    for (int f = 0; f < kTableMaxF; ++f) {
        const FeatureEntry &e = p.feat[f < p.n_features ? f : p.n_features - 1];
        out->fptr[f] = (const float *)p.base[e.target] + e.delta;
        out->raw8[f] = e.raw8;
    }
}

}  // namespace hpacml

namespace {

// Bytes a record of n rows x F words with row pitch ld (words) spans.
int64_t record_bytes(int64_t ld, int32_t F, int64_t n) { return n > 0 ? ((n - 1) * ld + F) * 4 : 0; }

// True when a record may share an element with a target the map reads.
bool record_overlaps_targets(const hpacml_map *m, const float *dst, int64_t ld, int32_t F, int64_t n) {
    const char *r0 = (const char *)dst, *r1 = r0 + record_bytes(ld, F, n);
    for (int t = 0; t < m->plan.n_targets; ++t) {
        const char *a0 = (const char *)m->plan.base[t];
        const char *a1 = a0 + 4 * (m->plan.max_elem[t] + 1);
        if (r0 < a1 && a0 < r1)
            return true;
    }
    return false;
}

// True when two records may share an element.  Interleaved records of one
// buffer (same pitch, disjoint column ranges, e.g. inputs in columns 0..8 and
// the output in column 9) are disjoint.
bool records_overlap(const float *a, int64_t lda, int32_t Fa, int64_t na, const float *b, int64_t ldb, int32_t Fb,
                     int64_t nb) {
    const char *a0 = (const char *)a, *a1 = a0 + record_bytes(lda, Fa, na);
    const char *b0 = (const char *)b, *b1 = b0 + record_bytes(ldb, Fb, nb);
    if (a1 <= b0 || b1 <= a0)
        return false;
    if (lda != ldb || (b0 - a0) % 4 != 0)
        return true;
    const int64_t d = (int64_t)(b0 - a0) / 4;
    int64_t r = d % lda;
    if (r < 0)
        r += lda;
    return !(Fa <= r && r + Fb <= lda);
}

// Validation shared by the collect entry points: shape, device, the record
// inside one device allocation and disjoint from what the map reads.
hpacml_status check_collect(const hpacml_map *m, float *dst, int64_t ld) {
    if (!m || !dst)
        return HPACML_E_INVAL;
    if (ld < m->plan.n_features)
        return HPACML_E_SHAPE;
    if (!same_device(m->device))
        return HPACML_E_INVAL;
    if (m->plan.n_points == 0)
        return HPACML_OK;
    hipDeviceptr_t abase = nullptr;
    size_t asize = 0;
    if (hipMemGetAddressRange(&abase, &asize, (hipDeviceptr_t)dst) != hipSuccess) {
        (void)hipGetLastError();
        return HPACML_E_INVAL;
    }
    const int64_t need = ((m->plan.n_points - 1) * ld + m->plan.n_features) * 4;
    if ((const char *)dst + need > (const char *)abase + asize || ((uintptr_t)dst & 3u))
        return HPACML_E_RANGE;
    if (record_overlaps_targets(m, dst, ld, m->plan.n_features, m->plan.n_points))
        return HPACML_E_ALIAS;
    return HPACML_OK;
}

// Hidden layers narrower than a fast kernel's uniform width H, zero-padded
// to it: the added neurons have zero weights and a zero bias, so their
// activation (ReLU or identity of 0) is 0 and, multiplied by the zero
// weights of the next layer, adds nothing to it; the padded model computes
// the unpadded one's sums (an infinite or NaN activation would turn a padded
// weight's 0 into NaN).  Returns false when a hidden layer is wider than H.
struct PaddedModel {
    std::vector<int32_t> dims;
    std::vector<std::vector<float>> W, b;
    std::vector<const float *> Wp, bp;
};
bool pad_hidden(int n_layers, const int32_t *dims, const float *const *W, const float *const *b, int H,
                PaddedModel &p) {
    p.dims.assign(dims, dims + n_layers + 1);
    for (int l = 1; l < n_layers; ++l) {
        if (dims[l] > H)
            return false;
        p.dims[l] = H;
    }
    p.W.assign(n_layers, {});
    p.b.assign(n_layers, {});
    p.Wp.assign(n_layers, nullptr);
    p.bp.assign(n_layers, nullptr);
    for (int l = 0; l < n_layers; ++l) {
        const int fi = dims[l], fo = dims[l + 1], pi = p.dims[l], po = p.dims[l + 1];
        p.W[l].assign((size_t)po * pi, 0.f);
        p.b[l].assign((size_t)po, 0.f);
        for (int o = 0; o < fo; ++o) {
            for (int i = 0; i < fi; ++i)
                p.W[l][(size_t)o * pi + i] = W[l][(size_t)o * fi + i];
            p.b[l][o] = b[l][o];
        }
        p.Wp[l] = p.W[l].data();
        p.bp[l] = p.b[l].data();
    }
    return true;
}

}  // namespace

extern "C" {

int32_t hpacml_abi_version(void) { return HPACML_ABI_VERSION; }

const char *hpacml_status_string(hpacml_status s) {
    switch (s) {
    case HPACML_OK: return "ok";
    case HPACML_E_INVAL: return "invalid argument";
    case HPACML_E_SHAPE: return "shape mismatch";
    case HPACML_E_RANGE: return "access out of range";
    case HPACML_E_ALIAS: return "output may overwrite an input before it is read";
    case HPACML_E_UNSUPPORTED: return "unsupported";
    case HPACML_E_NOMEM: return "out of memory";
    case HPACML_E_DEVICE: return "device error";
    }
    return "unknown status";
}

hpacml_status hpacml_map_validate(const hpacml_functor *f, int32_t dir, const hpacml_array *targets,
                                  int32_t n_targets, const hpacml_sweep *sweep, const int32_t *bnd,
                                  int64_t *n_points, int32_t *n_features) {
    try {
        MapPlan p;
        hpacml_status s = build_map_plan(f, dir, targets, n_targets, sweep, bnd, &p);
        if (s != HPACML_OK)
            return s;
        if (n_points)
            *n_points = p.n_points;
        if (n_features)
            *n_features = p.n_features;
        return HPACML_OK;
    } catch (const std::bad_alloc &) {
        return HPACML_E_NOMEM;
    } catch (...) {
        return HPACML_E_INVAL;
    }
}

void hpacml_map_destroy(hpacml_map *m) {
    if (!m)
        return;
    (void)hipFree(m->feat_dev);
    (void)hipFree(m->base_dev);
    (void)hipFree(m->stride_dev);
    (void)hipFree(m->tab_dev);
    hpacml_map_destroy(m->snap_map);
    (void)hipFree(m->snap);
    delete m;
}

hpacml_status hpacml_map_create(const hpacml_functor *f, int32_t dir, const hpacml_array *targets,
                                int32_t n_targets, const hpacml_sweep *sweep, const int32_t *bnd,
                                hpacml_map **out) {
    if (!out)
        return HPACML_E_INVAL;
    *out = nullptr;
    hpacml_map *m = nullptr;
    try {
        m = new hpacml_map_s();
        hpacml_status s = build_map_plan(f, dir, targets, n_targets, sweep, bnd, &m->plan);
        if (s == HPACML_OK && hipGetDevice(&m->device) != hipSuccess) {
            (void)hipGetLastError();
            s = HPACML_E_DEVICE;
        }
        if (s == HPACML_OK)
            s = check_device_targets(m->plan, m->device);
        if (s == HPACML_OK)
            s = upload(&m->feat_dev, m->plan.feat.data(), m->plan.feat.size());
        if (s == HPACML_OK) {
            std::vector<float *> bases(m->plan.n_targets);
            for (int t = 0; t < m->plan.n_targets; ++t)
                bases[t] = (float *)m->plan.base[t];
            s = upload(&m->base_dev, bases.data(), bases.size());
        }
        if (s == HPACML_OK)
            s = upload(&m->stride_dev, m->plan.stride.data(), m->plan.stride.size());
        if (s != HPACML_OK) {
            hpacml_map_destroy(m);
            return s;
        }
        m->dev = make_devmap(m->plan, m->feat_dev, m->base_dev, m->stride_dev);
        m->fast = make_map32(m->plan, &m->m32);
        m->t32 = table32_supported(m->plan, m->fast);
        if (m->t32) {
            table32_make(m->plan, &m->tab);
            s = upload(&m->tab_dev, &m->tab, 1);
            if (s != HPACML_OK) {
                hpacml_map_destroy(m);
                return s;
            }
        }
        *out = m;
        return HPACML_OK;
    } catch (const std::bad_alloc &) {
        hpacml_map_destroy(m);
        return HPACML_E_NOMEM;
    } catch (...) {
        hpacml_map_destroy(m);
        return HPACML_E_INVAL;
    }
}

hpacml_status hpacml_map_shape(const hpacml_map *m, int64_t *n_points, int32_t *n_features) {
    if (!m)
        return HPACML_E_INVAL;
    if (n_points)
        *n_points = m->plan.n_points;
    if (n_features)
        *n_features = m->plan.n_features;
    return HPACML_OK;
}

hpacml_status hpacml_model_validate(int32_t n_layers, const int32_t *dims, const int32_t *act,
                                    int32_t compute) {
    return validate_model(n_layers, dims, act, compute);
}

void hpacml_model_destroy(hpacml_model *m) {
    if (!m)
        return;
    (void)hipFree(m->gen_buf);
    (void)hipFree(m->f32_img);
    (void)hipFree(m->bf16_frags);
    (void)hipFree(m->bf16r_buf);
    (void)hipFree(m->cnn_buf);
    (void)hipFree(m->fused_buf);
    (void)hipFree(m->ws);
    layers_destroy(m->layers);
    delete m;
}

hpacml_status hpacml_model_create(int32_t n_layers, const int32_t *dims, const float *const *W,
                                  const float *const *b, const int32_t *act, int32_t compute,
                                  hpacml_model **out) {
    if (!out)
        return HPACML_E_INVAL;
    *out = nullptr;
    hpacml_status s = validate_model(n_layers, dims, act, compute);
    if (s != HPACML_OK)
        return s;
    if (!W || !b)
        return HPACML_E_INVAL;
    for (int l = 0; l < n_layers; ++l)
        if (!W[l] || !b[l])
            return HPACML_E_INVAL;
    hpacml_model *m = nullptr;
    try {
        m = new hpacml_model_s();
        m->n_layers = n_layers;
        m->compute = compute;
        m->dims.assign(dims, dims + n_layers + 1);
        m->act.assign(act, act + n_layers);
        if (hipGetDevice(&m->device) != hipSuccess) {
            (void)hipGetLastError();
            hpacml_model_destroy(m);
            return HPACML_E_DEVICE;
        }
        const bool bf16 = compute == HPACML_BF16;

        // general-shape layout: fp32 [out][in] per layer, then biases
        std::vector<float> hostw;
        std::vector<size_t> woff(n_layers), boff(n_layers);
        int maxw = 1;
        for (int l = 0; l < n_layers; ++l) {
            woff[l] = hostw.size();
            const size_t nw = (size_t)dims[l] * dims[l + 1];
            for (size_t i = 0; i < nw; ++i)
                hostw.push_back(bf16 ? host_bf16(W[l][i]) : W[l][i]);
            boff[l] = hostw.size();
            for (int o = 0; o < dims[l + 1]; ++o)
                hostw.push_back(b[l][o]);
        }
        for (int l = 0; l <= n_layers; ++l)
            maxw = dims[l] > maxw ? dims[l] : maxw;
        s = upload(&m->gen_buf, hostw.data(), hostw.size());
        if (s != HPACML_OK) {
            hpacml_model_destroy(m);
            return s;
        }
        {
            const hipError_t e = layers_create(n_layers, dims, act, W, b, compute, &m->layers);
            if (e != hipSuccess) {
                hpacml_model_destroy(m);
                return hip_status(e);
            }
        }
        m->gen.n_layers = n_layers;
        m->gen.bf16 = bf16 ? 1 : 0;
        m->gen.max_width = maxw;
        for (int l = 0; l <= n_layers; ++l)
            m->gen.dims[l] = dims[l];
        for (int l = 0; l < n_layers; ++l) {
            m->gen.act[l] = act[l];
            m->gen.W[l] = m->gen_buf + woff[l];
            m->gen.b[l] = m->gen_buf + boff[l];
        }

        // the fast kernels take uniform hidden widths; narrower or uneven
        // hidden layers run padded to the smallest width a kernel has
        int maxh = 0;
        for (int l = 1; l < n_layers; ++l)
            maxh = dims[l] > maxh ? dims[l] : maxh;
        const int H = bf16 ? (maxh <= 256 ? 256 : (maxh <= 512 ? 512 : 0))
                           : (maxh <= 64 ? 64 : (maxh <= 128 ? 128 : 0));
        PaddedModel pm;
        const int32_t *fd = dims;
        const float *const *fW = W;
        const float *const *fb = b;
        if (n_layers >= 2 && H > 0 && pad_hidden(n_layers, dims, W, b, H, pm)) {
            fd = pm.dims.data();
            fW = pm.Wp.data();
            fb = pm.bp.data();
            for (int l = 1; l < n_layers; ++l)
                m->padded = m->padded || dims[l] != H;
        }

        if (f32_fast_supported(n_layers, fd, compute)) {
            std::vector<float> img(f32_image_floats(n_layers, fd), 0.f);
            f32_pack(n_layers, fd, fW, fb, img.data());
            s = upload(&m->f32_img, img.data(), img.size());
            if (s != HPACML_OK) {
                hpacml_model_destroy(m);
                return s;
            }
            m->f32.hid = fd[1];
            m->f32.n_hidden = n_layers - 2;
            m->f32.ks1 = (fd[0] + 1) / 2;
            m->f32.f_out = fd[n_layers];
            for (int l = 0; l < n_layers; ++l)
                m->f32.act[l] = act[l];
            m->f32.lds_bytes = (int32_t)(img.size() * sizeof(float));
            m->f32.image = m->f32_img;
            m->variant = Variant::F32;
            m->fast_name = f32_variant_name(m->f32);
        } else if (bf16r_supported(n_layers, fd, act, compute)) {
            std::vector<uint8_t> buf;
            size_t off_w3 = 0, off_bias = 0;
            bf16r_pack(n_layers, fd, fW, fb, buf, &off_w3, &off_bias, &m->bf16r);
            s = upload(&m->bf16r_buf, buf.data(), buf.size());
            if (s != HPACML_OK) {
                hpacml_model_destroy(m);
                return s;
            }
            for (int l = 0; l < n_layers; ++l)
                m->bf16r.act[l] = act[l];
            m->bf16r.stream = m->bf16r_buf;
            m->bf16r.w3 = m->bf16r_buf + off_w3;
            m->bf16r.bias = (const float *)(m->bf16r_buf + off_bias);
            m->variant = Variant::BF16R;
            m->fast_name = bf16r_variant_name(m->bf16r);
        } else if (bf16_fast_supported(n_layers, fd, compute)) {
            std::vector<uint16_t> frags;
            bf16_pack(n_layers, fd, fW, fb, frags, &m->bf16);
            s = upload(&m->bf16_frags, frags.data(), frags.size());
            if (s != HPACML_OK) {
                hpacml_model_destroy(m);
                return s;
            }
            for (int l = 0; l < n_layers; ++l)
                m->bf16.act[l] = act[l];
            m->bf16.frags = m->bf16_frags;
            m->variant = Variant::BF16;
            m->fast_name = bf16_variant_name(m->bf16);
        }
        if (m->variant == Variant::Generic)
            m->padded = false;
        else if (m->padded)
            m->fast_name += "_padded";
        *out = m;
        return HPACML_OK;
    } catch (const std::bad_alloc &) {
        hpacml_model_destroy(m);
        return HPACML_E_NOMEM;
    } catch (...) {
        hpacml_model_destroy(m);
        return HPACML_E_INVAL;
    }
}

hpacml_status hpacml_cnn_validate(int32_t in_channels, int32_t height, int32_t width, int32_t n_layers,
                                  const hpacml_layer *layers, int32_t *out_shape) {
    CnnPlan p;
    hpacml_status s = validate_cnn(in_channels, height, width, n_layers, layers, &p);
    if (s == HPACML_OK && out_shape) {
        out_shape[0] = p.shape[n_layers].h;
        out_shape[1] = p.shape[n_layers].w;
        out_shape[2] = p.shape[n_layers].c;
    }
    return s;
}

hpacml_status hpacml_cnn_param_counts(int32_t in_channels, int32_t height, int32_t width, int32_t n_layers,
                                      const hpacml_layer *layers, int64_t *w_counts, int64_t *b_counts) {
    CnnPlan p;
    hpacml_status s = validate_cnn(in_channels, height, width, n_layers, layers, &p);
    if (s != HPACML_OK)
        return s;
    if (!w_counts || !b_counts)
        return HPACML_E_INVAL;
    for (int l = 0; l < n_layers; ++l) {
        const hpacml_layer &y = layers[l];
        const CnnShape &si = p.shape[l], &so = p.shape[l + 1];
        if (y.kind == HPACML_LAYER_CONV2D)
            w_counts[l] = (int64_t)so.c * si.c * y.kernel[0] * y.kernel[1];
        else if (y.kind == HPACML_LAYER_LINEAR)
            w_counts[l] = (int64_t)so.c * si.h * si.w * si.c;
        else
            w_counts[l] = 0;
        b_counts[l] = y.kind == HPACML_LAYER_MAXPOOL2D ? 0 : so.c;
    }
    return HPACML_OK;
}

hpacml_status hpacml_cnn_create(int32_t in_channels, int32_t height, int32_t width, int32_t n_layers,
                                const hpacml_layer *layers, const float *const *W, const float *const *b,
                                int32_t compute, hpacml_model **out) {
    if (!out)
        return HPACML_E_INVAL;
    *out = nullptr;
    CnnPlan p;
    hpacml_status s = validate_cnn(in_channels, height, width, n_layers, layers, &p);
    if (s != HPACML_OK)
        return s;
    if (compute != HPACML_F32)
        return HPACML_E_UNSUPPORTED;
    if (!W || !b)
        return HPACML_E_INVAL;
    for (int l = 0; l < n_layers; ++l)
        if (layers[l].kind != HPACML_LAYER_MAXPOOL2D && (!W[l] || !b[l]))
            return HPACML_E_INVAL;
    hpacml_model *m = nullptr;
    try {
        m = new hpacml_model_s();
        m->cnn = true;
        m->n_layers = n_layers;
        m->compute = compute;
        if (hipGetDevice(&m->device) != hipSuccess) {
            (void)hipGetLastError();
            hpacml_model_destroy(m);
            return HPACML_E_DEVICE;
        }
        // every layer's weights and biases: convolutions packed for the
        // layer kernel (32-byte aligned), fully connected layers in the
        // caller's layout
        std::vector<float> host;
        std::vector<size_t> woff(n_layers), boff(n_layers);
        for (int l = 0; l < n_layers; ++l) {
            const hpacml_layer &y = layers[l];
            const CnnShape &si = p.shape[l], &so = p.shape[l + 1];
            host.resize((host.size() + 7) / 8 * 8, 0.f);
            woff[l] = host.size();
            if (y.kind == HPACML_LAYER_CONV2D)
                cnn_conv_pack(W[l], so.c, si.c, y.kernel[0], y.kernel[1], host);
            else if (y.kind == HPACML_LAYER_LINEAR)
                host.insert(host.end(), W[l], W[l] + (size_t)so.c * si.h * si.w * si.c);
            boff[l] = host.size();
            if (y.kind != HPACML_LAYER_MAXPOOL2D)
                host.insert(host.end(), b[l], b[l] + so.c);
        }
        if (host.empty())
            host.push_back(0.f);   // a stack of pools only: no weights, a valid buffer all the same
        s = upload(&m->cnn_buf, host.data(), host.size());
        if (s == HPACML_OK && cnn_fused_supported(p)) {
            std::vector<float> packed;
            cnn_fused_pack(p, W, b, packed, &m->fused);
            s = upload(&m->fused_buf, packed.data(), packed.size());
            m->fused.wts = m->fused_buf;
            m->cnn_fused = true;
        }
        if (s != HPACML_OK) {
            hpacml_model_destroy(m);
            return s;
        }
        for (int l = 0; l < n_layers; ++l) {
            const hpacml_layer &y = layers[l];
            CnnLayerDev d{};
            d.kind = y.kind;
            d.cin = p.shape[l].c;
            d.cout = p.shape[l + 1].c;
            d.kh = y.kind == HPACML_LAYER_LINEAR ? 1 : y.kernel[0];
            d.kw = y.kind == HPACML_LAYER_LINEAR ? 1 : y.kernel[1];
            d.sh = y.kind == HPACML_LAYER_LINEAR ? 1 : y.stride[0];
            d.sw = y.kind == HPACML_LAYER_LINEAR ? 1 : y.stride[1];
            d.same = y.kind == HPACML_LAYER_CONV2D && y.padding == HPACML_PAD_SAME;
            d.mode = y.pad_mode;
            d.act = y.act;
            d.h = p.shape[l].h;
            d.w = p.shape[l].w;
            d.h2 = p.shape[l + 1].h;
            d.w2 = p.shape[l + 1].w;
            d.W = m->cnn_buf + woff[l];
            d.b = m->cnn_buf + boff[l];
            cnn_layer_divisors(d);
            m->cnn_layers.push_back(d);
        }
        m->cnnp = std::move(p);
        *out = m;
        return HPACML_OK;
    } catch (const std::bad_alloc &) {
        hpacml_model_destroy(m);
        return HPACML_E_NOMEM;
    } catch (...) {
        hpacml_model_destroy(m);
        return HPACML_E_INVAL;
    }
}

namespace {

bool maps_disjoint(const MapPlan &a, const MapPlan &b) {
    for (int i = 0; i < a.n_targets; ++i)
        for (int j = 0; j < b.n_targets; ++j)
            if (!disjoint_targets(a, i, b, j))
                return false;
    return true;
}

// (defined with the snapshot record below)
bool snapshot_t32(const hpacml_map *in);
hpacml_status take_snapshot(const hpacml_map *in, hipStream_t st, const hpacml_map **sm);

// The fused convolution kernel takes this call: 32-bit maps, outputs that
// meet no input (its tiles read their neighbours' pixels), and a tile that
// fits in LDS.
bool cnn_use_fused(const hpacml_model *model, const hpacml_map *in, const hpacml_map *out) {
    return model->cnn_fused && in->t32 && out->t32 && maps_disjoint(in->plan, out->plan) &&
           cnn_fused_tile_rows(model->fused, model->cnnp.height) > 0;
}

// Outputs that meet the inputs (a step written back into its own fields):
// the fused kernel still runs when it reads the inputs from the `to` map's
// snapshot record, filled first.
bool cnn_fused_on_snapshot(const hpacml_model *model, const hpacml_map *in, const hpacml_map *out) {
    return model->cnn_fused && in->t32 && out->t32 && !maps_disjoint(in->plan, out->plan) && snapshot_t32(in) &&
           cnn_fused_tile_rows(model->fused, model->cnnp.height) > 0;
}

hpacml_status cnn_infer(const hpacml_model *model, const hpacml_map *in, const hpacml_map *out, hipStream_t st) {
    const CnnPlan &c = model->cnnp;
    const int64_t S = in->plan.n_points / ((int64_t)c.height * c.width);
    if (S == 0)
        return HPACML_OK;   // no images: nothing to read or write
    if (cnn_use_fused(model, in, out))
        return hip_status(launch_cnn_fused(in->m32, out->m32, in->tab_dev, out->tab_dev, model->fused, (int32_t)S,
                                           c.height, c.width, st));
    if (cnn_fused_on_snapshot(model, in, out)) {
        const hpacml_map *sm = nullptr;
        hpacml_status s = take_snapshot(in, st, &sm);
        if (s != HPACML_OK)
            return s;
        return hip_status(launch_cnn_fused(sm->m32, out->m32, sm->tab_dev, out->tab_dev, model->fused, (int32_t)S,
                                           c.height, c.width, st));
    }
    // layer by layer: the first layer reads the map's tensor (the input
    // array itself when the map is a plain row-major view of it, else a
    // gathered copy in the workspace); the outputs are scattered after the
    // last layer, so they may overwrite inputs
    hpacml_model *mm = const_cast<hpacml_model *>(model);
    const int64_t per = (S * c.max_elems + 63) / 64 * 64;   // 256-byte aligned buffers
    // split-K partial sums of the fully connected layers
    int64_t part_floats = 0;
    for (const CnnLayerDev &L : model->cnn_layers) {
        const int z = linear_splits(L, S);
        if (z > 1)
            part_floats = std::max<int64_t>(part_floats, (int64_t)z * S * L.cout);
    }
    float *a = nullptr, *b = nullptr, *part = nullptr;
    {
        std::lock_guard<std::mutex> lock(mm->ws_mu);
        if (mm->ws_floats < 2 * per + part_floats) {
            float *buf = nullptr;
            hipError_t e = hipMalloc((void **)&buf, (size_t)(2 * per + part_floats) * sizeof(float));
            if (e != hipSuccess) {
                (void)hipGetLastError();
                return hip_status(e);
            }
            // the old workspace may still be in use by work queued on this stream
            e = hipStreamSynchronize(st);
            (void)hipFree(mm->ws);
            mm->ws = buf;
            mm->ws_floats = 2 * per + part_floats;
            if (e != hipSuccess)
                return hip_status(e);
        }
        a = mm->ws;
        b = mm->ws + per;
        part = mm->ws + 2 * per;
    }
    const float *x = a;
    if (in->plan.record_view) {
        x = (const float *)in->plan.base[0];
    } else {
        hpacml_status s = hpacml_collect(in, a, c.in_channels, st);
        if (s != HPACML_OK)
            return s;
    }
    const std::vector<CnnLayerDev> &ly = model->cnn_layers;
    const int tail = cnn_tail_start(ly);
    for (int l = 0; l < c.n_layers; ++l) {
        hipError_t e;
        if (l == tail) {
            // the closing fully connected layers and the scatter
            int splits = 1;
            e = launch_cnn_linear_partials(ly[l], x, b, S, part, &splits, st);
            if (e == hipSuccess)
                e = launch_cnn_tail(ly, l, splits > 1 ? part : b, splits, out->dev, S, st);
            return hip_status(e);
        }
        if (l + 1 < c.n_layers && cnn_pool_fusable(ly[l], ly[l + 1])) {
            e = launch_cnn_conv(ly[l], &ly[l + 1], x, b, S, st);   // convolution + max-pool
            ++l;
        } else {
            e = launch_cnn_layer(ly[l], x, b, S, part, st);
        }
        if (e != hipSuccess)
            return hip_status(e);
        x = b;
        std::swap(a, b);
    }
    return hip_status(launch_scatter_record(out->dev, x, st));
}

}  // namespace

namespace {

// The snapshot record of a TO map and the map that reads it back.  Feature-
// major ([F][B]: F targets of B points, so every element index stays below B
// and the map keeps the 32-bit form however large B * F is) when the `to` map
// itself has the 32-bit form (its collect can write that layout); otherwise
// row-major [B][F] read as one rank-2 target whose point b is the row
// (b, 0..F-1).
bool snapshot_feature_major(const hpacml_map *in) { return in->t32 && in->plan.n_features > 1; }

struct SnapshotDesc {
    hpacml_slice sl{};
    hpacml_functor fn{};
    std::vector<hpacml_array> a;
    hpacml_sweep sw{};
    int32_t bnd[HPACML_MAX_RANK] = {HPACML_BND_NONE, HPACML_BND_NONE, HPACML_BND_NONE, HPACML_BND_NONE};

    SnapshotDesc(int64_t B, int32_t F, float *buf, bool feature_major) {
        sw.step[0] = sw.step[1] = 1;
        sw.stop[0] = B;
        if (feature_major) {
            sl.count[0] = 1;
            fn = hpacml_functor{1, 1, &sl, F};
            a.resize(F);
            for (int f = 0; f < F; ++f) {
                a[f].data = buf + (size_t)f * B;
                a[f].dtype = HPACML_F32;
                a[f].extent[0] = B;
                a[f].stride[0] = 1;
            }
        } else {
            sl.count[0] = 1;
            sl.count[1] = F;
            fn = hpacml_functor{2, 1, &sl, F};
            a.resize(1);
            a[0].data = buf;
            a[0].dtype = HPACML_F32;
            a[0].extent[0] = B;
            a[0].extent[1] = F;
            a[0].stride[0] = F;
            a[0].stride[1] = 1;
            sw.stop[1] = 1;
        }
    }
};

// The snapshot record and its map, allocated on the first inference that
// needs them (the current device is the map's: check_infer has verified it).
hpacml_status snapshot_map(const hpacml_map *in, const hpacml_map **out) {
    std::lock_guard<std::mutex> lock(in->snap_mu);
    if (!in->snap_map) {
        const int64_t B = in->plan.n_points;
        const int32_t F = in->plan.n_features;
        float *buf = nullptr;
        hipError_t e = hipMalloc((void **)&buf, (size_t)B * F * sizeof(float));
        if (e != hipSuccess) {
            (void)hipGetLastError();
            return hip_status(e);
        }
        const SnapshotDesc d(B, F, buf, snapshot_feature_major(in));
        hpacml_map *m = nullptr;
        hpacml_status s =
            hpacml_map_create(&d.fn, HPACML_TO, d.a.data(), (int32_t)d.a.size(), &d.sw, d.bnd, &m);
        if (s != HPACML_OK) {
            (void)hipFree(buf);
            return s;
        }
        in->snap = buf;
        in->snap_map = m;
    }
    *out = in->snap_map;
    return HPACML_OK;
}

// Whether the snapshot map of `in` takes the 32-bit form, without allocating it.
bool snapshot_t32(const hpacml_map *in) {
    {
        std::lock_guard<std::mutex> lock(in->snap_mu);
        if (in->snap_map)
            return in->snap_map->t32;
    }
    // any non-null address serves the host-side plan
    const SnapshotDesc d(in->plan.n_points, in->plan.n_features, (float *)in->plan.base[0],
                         snapshot_feature_major(in));
    MapPlan p;
    Map32 m32;
    if (build_map_plan(&d.fn, HPACML_TO, d.a.data(), (int32_t)d.a.size(), &d.sw, d.bnd, &p) != HPACML_OK)
        return false;
    return table32_supported(p, make_map32(p, &m32));
}

// the kernel the dispatch below picks; `fast` = both maps take the 32-bit form
const char *kernel_name(const hpacml_model *model, bool fast, int64_t n_points) {
    if (fast && model->variant != Variant::Generic)
        return model->fast_name.c_str();
    if (layers_ready(model->layers, n_points))
        return layers_name(model->layers);
    return model->compute == HPACML_BF16 ? "mlp_generic_bf16" : "mlp_generic_f32";
}

// The general path of hpacml_infer: layer by layer through the matmul
// library, or the general fused kernel where the library has no algorithm.
hipError_t launch_general(const hpacml_model *model, const DevMap &in, const DevMap &out, hipStream_t st) {
    if (model->layers) {
        const hipError_t e = layers_infer(model->layers, in, out, st);
        if (e != hipErrorNotSupported)
            return e;
    }
    return launch_mlp_generic(in, out, model->gen, st);
}

// Every input of `in` into its snapshot record (stream-ordered before what
// follows); *sm = the map that reads the record.
hpacml_status take_snapshot(const hpacml_map *in, hipStream_t st, const hpacml_map **sm) {
    hpacml_status s = snapshot_map(in, sm);
    if (s != HPACML_OK)
        return s;
    if (snapshot_feature_major(in)) {
        CollectJob32 j = collect32_job(in->plan, in->m32, in->tab, in->tab_dev, (uint32_t *)in->snap, 1);
        j.dense = 0;
        j.fs = in->plan.n_points;
        return hip_status(launch_collect32(&j, 1, st));
    }
    return hpacml_collect(in, in->snap, in->plan.n_features, st);
}

// "snapshot+" prefixed names, kept for the life of the process
const char *snapshot_name(const char *kernel) {
    static std::mutex mu;
    static std::set<std::string> names;
    std::lock_guard<std::mutex> lock(mu);
    return names.insert(std::string("snapshot+") + kernel).first->c_str();
}

}  // namespace

namespace {

// ---- scratch for inference without allocation ------------------------------
// A fixed array per device holds the snapshot record of in-place inferences
// made through hpacml_infer_noalloc.  In host code `scratch` names a host-side
// stand-in: its device address comes from hipGetSymbolAddress, taken once per
// device (with that device current) and kept; only that address is ever
// passed to kernels.  Every call on a device shares the array, so calls that
// overlap on one device (different streams) race.
constexpr size_t kNoallocScratchBytes = HPACML_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

hpacml_status scratch_address(int device, void **out) {
    if (device < 0 || device >= kMaxDevices)
        return HPACML_E_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[device]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || p == nullptr) {
            (void)hipGetLastError();
            return HPACML_E_DEVICE;
        }
        g_scratch_ptr[device] = p;
    }
    *out = g_scratch_ptr[device];
    return HPACML_OK;
}

// The feature-major record [F][B] at `buf` as a rank-1 pointwise map in the
// 32-bit form: target f is buf + f * B, every feature reads its point.  Built
// without any allocation (no MapPlan); false when it does not fit the form.
bool record_map32(int64_t B, int32_t F, float *buf, Map32 *m, FeatTable32 *t) {
    if (B < 1 || B >= INT32_MAX / 3 || F < 1 || F > kTableMaxF)
        return false;
    Map32 r{};
    r.rank = 1;
    r.n_features = F;
    r.n_targets = F;
    r.n_points = (int32_t)B;
    for (int d = 0; d < HPACML_MAX_RANK; ++d) {
        r.count[d] = d == 0 ? (int32_t)B : 1;
        r.start[d] = 0;
        r.step[d] = 1;
        r.extent[d] = d == 0 ? (int32_t)B : 1;
        r.stride[d] = d == 0 ? 1 : 0;
        r.bnd[d] = HPACML_BND_NONE;
        r.omin[d] = r.omax[d] = 0;
        if (!set_div_magic(&r, d))
            return false;
    }
    for (int f = 0; f < kTableMaxF; ++f) {
        t->fptr[f] = buf + (size_t)(f < F ? f : F - 1) * B;
        t->raw8[f] = 0;
    }
    *m = r;
    return true;
}

}  // namespace

const char *hpacml_infer_variant(const hpacml_model *model, const hpacml_map *in, const hpacml_map *out) {
    bool snapshot = false;
    if (check_infer(model, in, out, &snapshot) != HPACML_OK)
        return nullptr;
    if (model->cnn)
        return cnn_use_fused(model, in, out)           ? "cnn_fused_f32"
               : cnn_fused_on_snapshot(model, in, out) ? "snapshot+cnn_fused_f32"
                                                       : "cnn_layers_f32";
    if (!snapshot)
        return kernel_name(model, in->t32 && out->t32, in->plan.n_points);
    return snapshot_name(kernel_name(model, snapshot_t32(in) && out->t32, in->plan.n_points));
}

hpacml_status hpacml_infer(const hpacml_model *model, const hpacml_map *in, const hpacml_map *out,
                           void *stream) {
    bool snapshot = false;
    hpacml_status s = check_infer(model, in, out, &snapshot);
    if (s != HPACML_OK)
        return s;
    if (in->plan.n_points == 0)
        return HPACML_OK;
    hipStream_t st = (hipStream_t)stream;
    if (model->cnn)
        return cnn_infer(model, in, out, st);
    if (snapshot) {
        // the outputs may overwrite elements that other points still read:
        // every point's inputs go to the snapshot record first, and the model
        // then reads them from there (stream order separates the two passes)
        const hpacml_map *sm = nullptr;
        s = take_snapshot(in, st, &sm);
        if (s != HPACML_OK)
            return s;
        in = sm;
    }
    hipError_t e;
    const bool fast = in->t32 && out->t32;
    switch (fast ? model->variant : Variant::Generic) {
    case Variant::F32: e = launch_mlp_f32(in->m32, out->m32, in->tab, out->tab, model->f32, st); break;
    case Variant::BF16: e = launch_mlp_bf16(in->m32, out->m32, in->tab, out->tab, model->bf16, st); break;
    case Variant::BF16R: e = launch_mlp_bf16r(in->m32, out->m32, in->tab, out->tab, model->bf16r, st); break;
    default: e = launch_general(model, in->dev, out->dev, st); break;
    }
    return hip_status(e);
}

hpacml_status hpacml_infer_noalloc(const hpacml_model *model, const hpacml_map *in, const hpacml_map *out,
                                   void *stream) {
    bool snapshot = false;
    hpacml_status s = check_infer(model, in, out, &snapshot);
    if (s != HPACML_OK)
        return s;
    if (model->cnn)
        return HPACML_E_UNSUPPORTED;
    hipStream_t st = (hipStream_t)stream;
    const bool fast = in->t32 && out->t32;
    if (!snapshot) {
        // disjoint (or element-for-element) maps: the kernels read the
        // application arrays directly and need no scratch
        if (in->plan.n_points == 0)
            return HPACML_OK;
        hipError_t e;
        switch (fast ? model->variant : Variant::Generic) {
        case Variant::F32: e = launch_mlp_f32(in->m32, out->m32, in->tab, out->tab, model->f32, st); break;
        case Variant::BF16: e = launch_mlp_bf16(in->m32, out->m32, in->tab, out->tab, model->bf16, st); break;
        case Variant::BF16R: e = launch_mlp_bf16r(in->m32, out->m32, in->tab, out->tab, model->bf16r, st); break;
        default: e = launch_mlp_generic(in->dev, out->dev, model->gen, st); break;
        }
        return hip_status(e);
    }
    // outputs that may overwrite inputs: the snapshot record goes to the
    // device's scratch array, read back through a map built on the host
    if (!fast || model->variant == Variant::Generic)
        return HPACML_E_UNSUPPORTED;
    const int64_t B = in->plan.n_points;
    const int32_t F = in->plan.n_features;
    if ((uint64_t)B * (uint64_t)F * sizeof(float) > kNoallocScratchBytes)
        return HPACML_E_RANGE;
    if (B == 0)
        return HPACML_OK;
    void *ptr = nullptr;
    s = scratch_address(model->device, &ptr);
    if (s != HPACML_OK)
        return s;
    Map32 rm{};
    FeatTable32 rt{};
    if (!record_map32(B, F, (float *)ptr, &rm, &rt))
        return HPACML_E_UNSUPPORTED;
    CollectJob32 j = collect32_job(in->plan, in->m32, in->tab, in->tab_dev, (uint32_t *)ptr, 1);
    j.dense = 0;
    j.fs = B;   // feature-major [F][B]
    hipError_t e = launch_collect32(&j, 1, st);
    if (e != hipSuccess)
        return hip_status(e);
    if (model->variant == Variant::F32)
        e = launch_mlp_f32(rm, out->m32, rt, out->tab, model->f32, st);
    else if (model->variant == Variant::BF16R)
        e = launch_mlp_bf16r(rm, out->m32, rt, out->tab, model->bf16r, st);
    else
        e = launch_mlp_bf16(rm, out->m32, rt, out->tab, model->bf16, st);
    return hip_status(e);
}

hpacml_status hpacml_collect(const hpacml_map *m, float *dst, int64_t ld, void *stream) {
    hpacml_status s = check_collect(m, dst, ld);
    if (s != HPACML_OK || m->plan.n_points == 0)
        return s;
    uint32_t *d = reinterpret_cast<uint32_t *>(dst);
    if (m->t32) {
        const CollectJob32 j = collect32_job(m->plan, m->m32, m->tab, m->tab_dev, d, ld);
        return hip_status(launch_collect32(&j, 1, (hipStream_t)stream));
    }
    return hip_status(launch_collect(m->dev, d, ld, (hipStream_t)stream));
}

hpacml_status hpacml_collect_pair(const hpacml_map *a, float *dst_a, int64_t ld_a, const hpacml_map *b, float *dst_b,
                                  int64_t ld_b, void *stream) {
    hpacml_status s = check_collect(a, dst_a, ld_a);
    if (s == HPACML_OK)
        s = check_collect(b, dst_b, ld_b);
    if (s != HPACML_OK)
        return s;
    if (a->device != b->device)
        return HPACML_E_INVAL;
    // the one launch reads both maps while it writes both records
    if (record_overlaps_targets(a, dst_b, ld_b, b->plan.n_features, b->plan.n_points) ||
        record_overlaps_targets(b, dst_a, ld_a, a->plan.n_features, a->plan.n_points) ||
        records_overlap(dst_a, ld_a, a->plan.n_features, a->plan.n_points, dst_b, ld_b, b->plan.n_features,
                        b->plan.n_points))
        return HPACML_E_ALIAS;
    uint32_t *da = reinterpret_cast<uint32_t *>(dst_a), *db = reinterpret_cast<uint32_t *>(dst_b);
    hipStream_t st = (hipStream_t)stream;
    if (a->t32 && b->t32) {
        CollectJob32 j[2];
        int n = 0;
        if (a->plan.n_points > 0)
            j[n++] = collect32_job(a->plan, a->m32, a->tab, a->tab_dev, da, ld_a);
        if (b->plan.n_points > 0)
            j[n++] = collect32_job(b->plan, b->m32, b->tab, b->tab_dev, db, ld_b);
        return n == 0 ? HPACML_OK : hip_status(launch_collect32(j, n, st));
    }
    // maps outside the 32-bit form: two launches, same result
    s = hpacml_collect(a, dst_a, ld_a, stream);
    return s == HPACML_OK ? hpacml_collect(b, dst_b, ld_b, stream) : s;
}

}  // extern "C"
