/* The C ABI used from plain C (C99, no C++ and no Python): a pointwise map
 * over three device arrays, a two-layer model whose result is exact in fp32
 * for the small-integer inputs used here (relu(x0) + relu(x1) + relu(x2)),
 * inference through a `from` map, and a collect record of the inputs.
 * Prints "ok" and exits 0 when every output and every recorded bit matches. */
#include <hip/hip_runtime_api.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "hpacml.h"

#define N 10007

static int fail(const char *what, int code) {
    fprintf(stderr, "%s failed: %s (%d)\n", what, code >= 0 ? hpacml_status_string((hpacml_status)code) : "hip", code);
    return 1;
}

int main(void) {
    float *host_in[3], *dev_in[3], *dev_out, *dev_rec;
    for (int t = 0; t < 3; ++t) {
        host_in[t] = (float *)malloc(N * sizeof(float));
        for (int i = 0; i < N; ++i)
            host_in[t][i] = (float)((i * (t + 3)) % 17 - 8);   /* small integers, some negative */
        if (hipMalloc((void **)&dev_in[t], N * sizeof(float)) != hipSuccess)
            return fail("hipMalloc", -1);
        hipMemcpy(dev_in[t], host_in[t], N * sizeof(float), hipMemcpyHostToDevice);
    }
    if (hipMalloc((void **)&dev_out, N * sizeof(float)) != hipSuccess ||
        hipMalloc((void **)&dev_rec, 3 * N * sizeof(float)) != hipSuccess)
        return fail("hipMalloc", -1);

    /* [i, 0:3] = ([i]) over three arrays; [i, 0:1] = ([i]) over one */
    hpacml_slice sl;
    memset(&sl, 0, sizeof sl);
    sl.count[0] = 1;
    hpacml_functor fin = {1, 1, &sl, 3}, fout = {1, 1, &sl, 1};
    hpacml_array arr[3], oarr;
    memset(arr, 0, sizeof arr);
    memset(&oarr, 0, sizeof oarr);
    for (int t = 0; t < 3; ++t) {
        arr[t].data = dev_in[t];
        arr[t].dtype = HPACML_F32;
        arr[t].extent[0] = N;
        arr[t].stride[0] = 1;
    }
    oarr = arr[0];
    oarr.data = dev_out;
    hpacml_sweep sw;
    memset(&sw, 0, sizeof sw);
    sw.stop[0] = N;
    sw.step[0] = 1;
    int32_t bnd[HPACML_MAX_RANK] = {HPACML_BND_NONE, HPACML_BND_NONE, HPACML_BND_NONE, HPACML_BND_NONE};
    hpacml_map *in = NULL, *out = NULL;
    hpacml_status s = hpacml_map_create(&fin, HPACML_TO, arr, 3, &sw, bnd, &in);
    if (s != HPACML_OK)
        return fail("hpacml_map_create(to)", s);
    s = hpacml_map_create(&fout, HPACML_FROM, &oarr, 1, &sw, bnd, &out);
    if (s != HPACML_OK)
        return fail("hpacml_map_create(from)", s);

    /* 3 -> 4 (identity rows + a zero row, ReLU) -> 1 (sum of the first three) */
    const float W1[12] = {1, 0, 0, 0, 1, 0, 0, 0, 1, 0, 0, 0}, b1[4] = {0, 0, 0, 0};
    const float W2[4] = {1, 1, 1, 0}, b2[1] = {0};
    const float *W[2] = {W1, W2}, *b[2] = {b1, b2};
    const int32_t dims[3] = {3, 4, 1}, act[2] = {HPACML_ACT_RELU, HPACML_ACT_IDENTITY};
    hpacml_model *model = NULL;
    s = hpacml_model_create(2, dims, W, b, act, HPACML_F32, &model);
    if (s != HPACML_OK)
        return fail("hpacml_model_create", s);

    s = hpacml_infer(model, in, out, NULL);
    if (s != HPACML_OK)
        return fail("hpacml_infer", s);
    s = hpacml_collect(in, dev_rec, 3, NULL);
    if (s != HPACML_OK)
        return fail("hpacml_collect", s);
    if (hipDeviceSynchronize() != hipSuccess)
        return fail("hipDeviceSynchronize", -1);

    float *got = (float *)malloc(N * sizeof(float)), *rec = (float *)malloc(3 * N * sizeof(float));
    hipMemcpy(got, dev_out, N * sizeof(float), hipMemcpyDeviceToHost);
    hipMemcpy(rec, dev_rec, 3 * N * sizeof(float), hipMemcpyDeviceToHost);
    int bad = 0;
    for (int i = 0; i < N; ++i) {
        float want = 0.f;
        for (int t = 0; t < 3; ++t) {
            want += host_in[t][i] > 0.f ? host_in[t][i] : 0.f;
            if (memcmp(&rec[3 * i + t], &host_in[t][i], sizeof(float)) != 0)
                ++bad;
        }
        if (got[i] != want)
            ++bad;
    }
    printf("%s: %d points, kernel %s, %d mismatches\n", bad ? "FAIL" : "ok", N, hpacml_infer_variant(model, in, out),
           bad);
    hpacml_model_destroy(model);
    hpacml_map_destroy(in);
    hpacml_map_destroy(out);
    return bad ? 1 : 0;
}
