// Execution control of a region (Sec. III-C, Fig. 3 `ml(infer | collect |
// predicated)` and `if`; Sec. IV-B): per invocation, inference, or data
// collection around the accurate path, and the sink the collected samples go
// to (one region group of the database: inputs, outputs, region time).
//
// Host code over the public entry points: inference is hpacml_infer, the
// records are hpacml_collect of the `to` map before and of the `from` map
// after the accurate path, straight into the sample's slot of the sink.
#include <hip/hip_runtime.h>

#include <cerrno>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <sys/stat.h>
#include <vector>

#include "hpacml.h"
#include "kernels.hpp"

struct hpacml_region_s {
    const hpacml_map *in = nullptr, *out = nullptr;
    const hpacml_model *model = nullptr;
    int32_t mode = 0;
    int64_t points = 0, points_out = 0;   // rows of the two datasets' samples
    int32_t f_in = 0, f_out = 0;
    int64_t capacity = 0, n = 0;
    float *in_rec = nullptr, *out_rec = nullptr;   // device [capacity][points][F]
    std::vector<hipEvent_t> ev;                    // [3 * capacity]: around each accurate path, and
                                                   // after the sample's output record
    std::mutex mu;
};

namespace {

hpacml_status hip_status(hipError_t e) {
    if (e == hipSuccess)
        return HPACML_OK;
    (void)hipGetLastError();
    return e == hipErrorOutOfMemory ? HPACML_E_NOMEM : HPACML_E_DEVICE;
}

// NumPy .npy, version 1.0: magic, version, header length, a Python dict
// literal padded with spaces to a 64-byte boundary and ending in '\n', data.
bool write_npy(const std::string &path, const float *data, const std::vector<int64_t> &shape) {
    std::string dims;
    for (size_t i = 0; i < shape.size(); ++i)
        dims += std::to_string(shape[i]) + (shape.size() == 1 || i + 1 < shape.size() ? "," : "");
    std::string hdr = "{'descr': '<f4', 'fortran_order': False, 'shape': (" + dims + "), }";
    const size_t pre = 10;   // magic (6) + version (2) + header length (2)
    while ((pre + hdr.size() + 1) % 64)
        hdr += ' ';
    hdr += '\n';
    FILE *f = std::fopen(path.c_str(), "wb");
    if (!f)
        return false;
    const unsigned char head[8] = {0x93, 'N', 'U', 'M', 'P', 'Y', 1, 0};
    const uint16_t len = (uint16_t)hdr.size();
    const unsigned char lb[2] = {(unsigned char)(len & 0xFF), (unsigned char)(len >> 8)};
    size_t count = 1;
    for (int64_t d : shape)
        count *= (size_t)d;
    bool ok = std::fwrite(head, 1, 8, f) == 8 && std::fwrite(lb, 1, 2, f) == 2 &&
              std::fwrite(hdr.data(), 1, hdr.size(), f) == hdr.size() &&
              (count == 0 || std::fwrite(data, sizeof(float), count, f) == count);
    ok = (std::fclose(f) == 0) && ok;
    return ok;
}

bool make_dir(const std::string &d) { return ::mkdir(d.c_str(), 0755) == 0 || errno == EEXIST; }

// Record one map into the sample slot `dst` ([points][F], ld = F).
hpacml_status record(const hpacml_map *m, float *dst, int32_t F, void *stream) {
    return hpacml_collect(m, dst, F, stream);
}

}  // namespace

extern "C" {

hpacml_status hpacml_region_create(const hpacml_model *model, const hpacml_map *in, const hpacml_map *out,
                                   int32_t mode, int64_t capacity, hpacml_region **region) {
    if (!region)
        return HPACML_E_INVAL;
    *region = nullptr;
    if (mode < HPACML_MODE_INFER || mode > HPACML_MODE_PREDICATED || capacity < 0)
        return HPACML_E_INVAL;
    hpacml_status s = hpacml::infer_status(model, in, out);
    if (s != HPACML_OK)
        return s;
    hpacml_region *r = nullptr;
    try {
        r = new hpacml_region_s();
        r->in = in;
        r->out = out;
        r->model = model;
        r->mode = mode;
        hpacml_map_shape(in, &r->points, &r->f_in);
        hpacml_map_shape(out, &r->points_out, &r->f_out);
        r->capacity = mode == HPACML_MODE_INFER ? 0 : capacity;
        if (r->capacity > 0 && r->points > 0) {
            const size_t n_in = (size_t)r->capacity * r->points * r->f_in;
            const size_t n_out = (size_t)r->capacity * r->points_out * r->f_out;
            hipError_t e = hipMalloc((void **)&r->in_rec, n_in * sizeof(float));
            if (e == hipSuccess)
                e = hipMalloc((void **)&r->out_rec, n_out * sizeof(float));
            if (e != hipSuccess) {
                hpacml_region_destroy(r);
                return hip_status(e);
            }
        }
        r->ev.assign((size_t)(3 * r->capacity), nullptr);
        *region = r;
        return HPACML_OK;
    } catch (const std::bad_alloc &) {
        hpacml_region_destroy(r);
        return HPACML_E_NOMEM;
    }
}

hpacml_status hpacml_region_run(hpacml_region *r, int32_t cond, int32_t enabled, hpacml_accurate_fn accurate,
                                void *user, void *stream) {
    if (!r)
        return HPACML_E_INVAL;
    hipStream_t st = (hipStream_t)stream;
    if (!enabled) {
        // if(false): the original code only
        if (!accurate)
            return HPACML_E_INVAL;
        accurate(user, stream);
        return hip_status(hipGetLastError());
    }
    const bool infer = r->mode == HPACML_MODE_INFER || (r->mode == HPACML_MODE_PREDICATED && cond != 0);
    if (infer)
        return hpacml_infer(r->model, r->in, r->out, stream);
    if (!accurate)
        return HPACML_E_INVAL;
    std::lock_guard<std::mutex> lock(r->mu);
    if (r->n >= r->capacity)
        return HPACML_E_RANGE;
    const int64_t k = r->n;
    float *in_slot = r->in_rec ? r->in_rec + (size_t)k * r->points * r->f_in : nullptr;
    float *out_slot = r->out_rec ? r->out_rec + (size_t)k * r->points_out * r->f_out : nullptr;
    hipEvent_t &e0 = r->ev[3 * k], &e1 = r->ev[3 * k + 1], &e2 = r->ev[3 * k + 2];
    hipError_t he = hipSuccess;
    if (!e0)
        he = hipEventCreate(&e0);
    if (he == hipSuccess && !e1)
        he = hipEventCreate(&e1);
    if (he == hipSuccess && !e2)
        he = hipEventCreateWithFlags(&e2, hipEventDisableTiming);
    if (he != hipSuccess)
        return hip_status(he);
    // inputs before the accurate path writes anything, outputs after it
    hpacml_status s = r->points ? record(r->in, in_slot, r->f_in, stream) : HPACML_OK;
    if (s != HPACML_OK)
        return s;
    if ((he = hipEventRecord(e0, st)) != hipSuccess)
        return hip_status(he);
    accurate(user, stream);
    if ((he = hipEventRecord(e1, st)) != hipSuccess)
        return hip_status(he);
    s = r->points_out ? record(r->out, out_slot, r->f_out, stream) : HPACML_OK;
    if (s != HPACML_OK)
        return s;
    // the sample is complete once this event has passed (read waits on it)
    if ((he = hipEventRecord(e2, st)) != hipSuccess)
        return hip_status(he);
    r->n = k + 1;
    return HPACML_OK;
}

hpacml_status hpacml_region_samples(const hpacml_region *r, int64_t *n) {
    if (!r || !n)
        return HPACML_E_INVAL;
    *n = r->n;
    return HPACML_OK;
}

hpacml_status hpacml_region_read(const hpacml_region *r, int64_t n, float *inputs, float *outputs,
                                 float *times_ms) {
    if (!r || n < 0)
        return HPACML_E_INVAL;
    if (n > r->n)
        return HPACML_E_RANGE;
    hipError_t e = hipSuccess;
    // every sample's records complete, whatever stream the region ran on
    // (a blocking copy is ordered after the null stream only)
    for (int64_t k = 0; e == hipSuccess && k < n; ++k)
        e = hipEventSynchronize(r->ev[3 * k + 2]);
    if (e == hipSuccess && inputs && n && r->points)
        e = hipMemcpy(inputs, r->in_rec, (size_t)n * r->points * r->f_in * sizeof(float), hipMemcpyDeviceToHost);
    if (e == hipSuccess && outputs && n && r->points_out)
        e = hipMemcpy(outputs, r->out_rec, (size_t)n * r->points_out * r->f_out * sizeof(float),
                      hipMemcpyDeviceToHost);
    for (int64_t k = 0; e == hipSuccess && times_ms && k < n; ++k) {
        e = hipEventElapsedTime(&times_ms[k], r->ev[3 * k], r->ev[3 * k + 1]);
    }
    return hip_status(e);
}

hpacml_status hpacml_region_save(const hpacml_region *r, const char *dir, const char *name) {
    if (!r || !dir || !name || !*name || std::strchr(name, '/'))
        return HPACML_E_INVAL;
    try {
        const int64_t n = r->n;
        std::vector<float> in((size_t)n * r->points * r->f_in), out((size_t)n * r->points_out * r->f_out);
        std::vector<float> t((size_t)n);
        hpacml_status s = hpacml_region_read(r, n, in.data(), out.data(), t.data());
        if (s != HPACML_OK)
            return s;
        const std::string group = std::string(dir) + "/" + name;
        if (!make_dir(dir) || !make_dir(group))
            return HPACML_E_INVAL;
        if (!write_npy(group + "/inputs.npy", in.data(), {n, r->points, r->f_in}) ||
            !write_npy(group + "/outputs.npy", out.data(), {n, r->points_out, r->f_out}) ||
            !write_npy(group + "/time.npy", t.data(), {n}))
            return HPACML_E_INVAL;
        return HPACML_OK;
    } catch (const std::bad_alloc &) {
        return HPACML_E_NOMEM;
    }
}

hpacml_status hpacml_region_reset(hpacml_region *r) {
    if (!r)
        return HPACML_E_INVAL;
    std::lock_guard<std::mutex> lock(r->mu);
    r->n = 0;
    return HPACML_OK;
}

void hpacml_region_destroy(hpacml_region *r) {
    if (!r)
        return;
    for (hipEvent_t e : r->ev)
        if (e)
            (void)hipEventDestroy(e);
    (void)hipFree(r->in_rec);
    (void)hipFree(r->out_rec);
    delete r;
}

}  // extern "C"
