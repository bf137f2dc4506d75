// Host-side access plan of a tensor map: descriptor validation plus the
// extraction / resolution / wrapping steps of the data bridge (Sec. IV-A).
#include "plan.hpp"

#include <algorithm>
#include <climits>

namespace hpacml {

namespace {

constexpr int64_t kMaxExtent = int64_t(1) << 40;

bool mul_ok(int64_t a, int64_t b, int64_t *r) { return !__builtin_mul_overflow(a, b, r); }
bool add_ok(int64_t a, int64_t b, int64_t *r) { return !__builtin_add_overflow(a, b, r); }

int64_t ceil_div(int64_t a, int64_t b) { return a <= 0 ? 0 : (a + b - 1) / b; }

int64_t pos_mod(int64_t x, int64_t n) {
    int64_t r = x % n;
    return r < 0 ? r + n : r;
}

// Sufficient test that distinct sweep points address distinct elements of a
// target.  Along dimension d the resolved coordinates of the points are
// distinct values in [0, extent) (a periodic shift permutes them, a clamped
// `from` map has no offset), spanning at most `span_d`: (count-1)*step without
// a wrap, extent-1 with one.  Visiting the swept dimensions by increasing
// stride, each stride must exceed the largest element distance the finer
// dimensions can produce, sum(stride * span); then two points that differ in
// their coarsest differing dimension cannot meet.  Row-major and strided views
// pass; a zero stride or a stride that folds the sweep does not.
bool injective_sweep(const MapPlan &p, const hpacml_array &a) {
    struct Dim {
        int64_t stride, span;
    };
    Dim dims[HPACML_MAX_RANK];
    int n = 0;
    for (int d = 0; d < p.rank; ++d) {
        if (p.count[d] <= 1)
            continue;
        int64_t span = (p.count[d] - 1) * p.step[d];
        const int64_t first = p.start[d] + p.raw[d], last = first + span;   // slice 0 of the functor
        if (p.bnd[d] == HPACML_BND_PERIODIC && (first < 0 || last >= p.extent[d]))
            span = p.extent[d] - 1;
        dims[n++] = {a.stride[d], span};
    }
    std::sort(dims, dims + n, [](const Dim &x, const Dim &y) { return x.stride < y.stride; });
    int64_t reach = 0;   // largest element distance of the finer dimensions
    for (int i = 0; i < n; ++i) {
        if (dims[i].stride <= reach)
            return false;
        int64_t term;
        if (!mul_ok(dims[i].stride, dims[i].span, &term) || !add_ok(reach, term, &reach))
            return false;
    }
    return true;
}

}  // namespace

hpacml_status build_map_plan(const hpacml_functor *f, int32_t dir, const hpacml_array *targets,
                             int32_t n_targets, const hpacml_sweep *sweep, const int32_t *bnd,
                             MapPlan *out) {
    if (!f || !targets || !sweep || !bnd || !out)
        return HPACML_E_INVAL;
    if (dir != HPACML_TO && dir != HPACML_FROM)
        return HPACML_E_INVAL;
    const int R = f->rank;
    if (R < 1 || R > HPACML_MAX_RANK)
        return HPACML_E_INVAL;
    if (f->n_slices < 1 || !f->slices)
        return HPACML_E_INVAL;
    if (f->n_slices > HPACML_MAX_SLICES)
        return HPACML_E_UNSUPPORTED;
    if (n_targets < 1)
        return HPACML_E_INVAL;
    if (n_targets > HPACML_MAX_TARGETS)
        return HPACML_E_UNSUPPORTED;

    // functor: feature count per target = sum over slices of prod(count)
    int64_t per_target = 0;
    for (int s = 0; s < f->n_slices; ++s) {
        int64_t e = 1;
        for (int d = 0; d < R; ++d) {
            int32_t c = f->slices[s].count[d];
            if (c < 1)
                return HPACML_E_INVAL;
            if (!mul_ok(e, c, &e) || e > (int64_t)HPACML_MAX_FEATURES * HPACML_MAX_TARGETS)
                return HPACML_E_UNSUPPORTED;
        }
        per_target += e;
    }
    if (per_target * n_targets != (int64_t)f->n_features)
        return HPACML_E_SHAPE;
    if (f->n_features > HPACML_MAX_FEATURES)
        return HPACML_E_UNSUPPORTED;

    // `from` maps write one element per target per point (the paper's only
    // `from` functor is [i, j, 0:1] = ([i, j]), Fig. 2)
    if (dir == HPACML_FROM) {
        if (f->n_slices != 1)
            return HPACML_E_UNSUPPORTED;
        for (int d = 0; d < R; ++d)
            if (f->slices[0].count[d] != 1)
                return HPACML_E_UNSUPPORTED;
    }

    // targets: one shared index space, f32 elements, non-negative strides
    for (int t = 0; t < n_targets; ++t) {
        const hpacml_array &a = targets[t];
        if (!a.data || a.reserved != 0)
            return HPACML_E_INVAL;
        if (a.dtype != HPACML_F32)
            return HPACML_E_UNSUPPORTED;
        for (int d = 0; d < R; ++d) {
            if (a.extent[d] < 1 || a.stride[d] < 0)
                return HPACML_E_INVAL;
            if (a.extent[d] > kMaxExtent || a.stride[d] > kMaxExtent)
                return HPACML_E_UNSUPPORTED;
            if (a.extent[d] != targets[0].extent[d])
                return HPACML_E_SHAPE;
        }
    }

    MapPlan p;
    p.rank = R;
    p.dir = dir;
    p.n_targets = n_targets;
    p.n_features = f->n_features;

    // sweep and boundary modes
    int64_t npts = 1;
    for (int d = 0; d < R; ++d) {
        if (bnd[d] < HPACML_BND_NONE || bnd[d] > HPACML_BND_CLAMP)
            return HPACML_E_INVAL;
        if (sweep->step[d] < 1)
            return HPACML_E_INVAL;
        const int64_t n = targets[0].extent[d];
        if (sweep->start[d] < 0 || sweep->start[d] > sweep->stop[d] || sweep->stop[d] > n)
            return HPACML_E_RANGE;
        p.extent[d] = n;
        p.start[d] = sweep->start[d];
        p.step[d] = sweep->step[d];
        p.count[d] = ceil_div(sweep->stop[d] - sweep->start[d], sweep->step[d]);
        p.bnd[d] = bnd[d];
        if (!mul_ok(npts, p.count[d], &npts))
            return HPACML_E_UNSUPPORTED;
    }
    p.n_points = npts;

    // extraction + resolution: raw offset of every feature's element
    p.raw.assign((size_t)p.n_features * 4, 0);
    {
        int fi = 0;
        for (int t = 0; t < n_targets; ++t)
            for (int s = 0; s < f->n_slices; ++s) {
                const hpacml_slice &sl = f->slices[s];
                int64_t total = 1;
                for (int d = 0; d < R; ++d)
                    total *= sl.count[d];
                for (int64_t e = 0; e < total; ++e) {
                    int64_t rem = e, ed[HPACML_MAX_RANK] = {0, 0, 0, 0};
                    for (int d = R - 1; d >= 0; --d) {
                        ed[d] = rem % sl.count[d];
                        rem /= sl.count[d];
                    }
                    for (int d = 0; d < R; ++d) {
                        int64_t o = (int64_t)sl.lo[d] + ed[d];
                        if (o < INT32_MIN || o > INT32_MAX)
                            return HPACML_E_UNSUPPORTED;
                        p.raw[(size_t)fi * 4 + d] = (int32_t)o;
                    }
                    ++fi;
                }
            }
    }
    p.pointwise = true;
    for (int d = 0; d < R; ++d) {
        int32_t lo = INT32_MAX, hi = INT32_MIN;
        for (int fi = 0; fi < p.n_features; ++fi) {
            lo = std::min(lo, p.raw[(size_t)fi * 4 + d]);
            hi = std::max(hi, p.raw[(size_t)fi * 4 + d]);
        }
        p.omin[d] = lo;
        p.omax[d] = hi;
        if (lo != 0 || hi != 0)
            p.pointwise = false;
    }

    // accesses outside [0, extent) need a boundary mode
    if (npts > 0)
        for (int d = 0; d < R; ++d) {
            if (p.bnd[d] != HPACML_BND_NONE)
                continue;
            int64_t first = p.start[d] + p.omin[d];
            int64_t last = p.start[d] + (p.count[d] - 1) * p.step[d] + p.omax[d];
            if (first < 0 || last >= p.extent[d])
                return HPACML_E_RANGE;
        }

    // a clamped `from` offset would make two points write one element
    if (dir == HPACML_FROM)
        for (int d = 0; d < R; ++d)
            if (p.bnd[d] == HPACML_BND_CLAMP && f->slices[0].lo[d] != 0)
                return HPACML_E_INVAL;

    // a `from` map writes one element per point and target, so two sweep
    // points must never land on one element: stride-0 views (broadcasts) and
    // strides that fold the sweep onto itself are refused
    if (dir == HPACML_FROM && npts > 1)
        for (int t = 0; t < n_targets; ++t)
            if (!injective_sweep(p, targets[t]))
                return HPACML_E_ALIAS;

    // wrapping: per-target base and strides, element extents
    p.base.resize(n_targets);
    p.stride.assign((size_t)n_targets * 4, 0);
    p.max_elem.resize(n_targets);
    p.idx32 = true;
    for (int t = 0; t < n_targets; ++t) {
        p.base[t] = targets[t].data;
        int64_t m = 0;
        for (int d = 0; d < R; ++d) {
            p.stride[(size_t)t * 4 + d] = targets[t].stride[d];
            int64_t term;
            if (!mul_ok(p.extent[d] - 1, targets[t].stride[d], &term) || !add_ok(m, term, &m))
                return HPACML_E_UNSUPPORTED;
        }
        p.max_elem[t] = m;
        if (m > INT32_MAX)
            p.idx32 = false;
    }

    // per-feature table for the kernels
    p.feat.resize(p.n_features);
    p.raw8 = true;
    {
        int fi = 0;
        for (int t = 0; t < n_targets; ++t)
            for (int k = 0; k < p.n_features / n_targets; ++k, ++fi) {
                FeatureEntry &e = p.feat[fi];
                e.target = t;
                e.raw8 = 0;
                int64_t delta = 0;
                for (int d = 0; d < HPACML_MAX_RANK; ++d) {
                    int64_t o = d < R ? p.raw[(size_t)fi * 4 + d] : 0;
                    if (o < -127 || o > 127 || (p.bnd[d] == HPACML_BND_PERIODIC && (o > p.extent[d] || -o > p.extent[d])))
                        p.raw8 = false;
                    else
                        e.raw8 |= (uint32_t)(uint8_t)(int8_t)o << (8 * d);
                    if (d < R && p.bnd[d] == HPACML_BND_PERIODIC)
                        e.off[d] = (int32_t)pos_mod(o, p.extent[d]);
                    else
                        e.off[d] = (int32_t)o;
                    if (d < R)
                        delta += o * p.stride[(size_t)t * 4 + d];
                }
                e.delta = delta;
            }
    }

    // is the map's tensor [points][features] target 0's memory itself?  One
    // target, every access inside the array (no boundary mode applies), the
    // sweep's first point at element 0, feature f at element offset f, and
    // the point strides those of a row-major [count...][F] array.
    p.record_view = n_targets == 1 && npts > 0;
    if (p.record_view) {
        int64_t e0 = 0;
        for (int d = 0; d < R; ++d) {
            if (p.start[d] + p.omin[d] < 0 ||
                p.start[d] + (p.count[d] - 1) * p.step[d] + p.omax[d] >= p.extent[d])
                p.record_view = false;
            e0 += p.start[d] * p.stride[d];
        }
        for (int fi = 0; p.record_view && fi < p.n_features; ++fi)
            p.record_view = e0 + p.feat[fi].delta == fi;
        int64_t want = p.n_features;
        for (int d = R - 1; p.record_view && d >= 0; --d) {
            if (p.count[d] > 1 && p.step[d] * p.stride[d] != want)
                p.record_view = false;
            want *= p.count[d];
        }
    }
    *out = std::move(p);
    return HPACML_OK;
}

hpacml_status validate_model(int32_t n_layers, const int32_t *dims, const int32_t *act,
                             int32_t compute) {
    if (!dims || !act)
        return HPACML_E_INVAL;
    if (n_layers < 1)
        return HPACML_E_INVAL;
    if (n_layers > HPACML_MAX_LAYERS)
        return HPACML_E_UNSUPPORTED;
    if (compute != HPACML_F32 && compute != HPACML_BF16)
        return HPACML_E_INVAL;
    for (int l = 0; l <= n_layers; ++l) {
        if (dims[l] < 1)
            return HPACML_E_INVAL;
        if (dims[l] > HPACML_MAX_WIDTH)
            return HPACML_E_UNSUPPORTED;
    }
    if (dims[0] > HPACML_MAX_FEATURES || dims[n_layers] > HPACML_MAX_TARGETS)
        return HPACML_E_UNSUPPORTED;
    for (int l = 0; l < n_layers; ++l)
        if (act[l] != HPACML_ACT_IDENTITY && act[l] != HPACML_ACT_RELU)
            return HPACML_E_INVAL;
    return HPACML_OK;
}

// Element sets of two targets are disjoint when they share strides, every
// stride is a multiple of the smallest non-zero stride s, and the bases differ
// by a whole number of elements that is not a multiple of s (interleaved
// fields of one array of structures), or when their byte ranges do not meet.
bool disjoint_targets(const MapPlan &a, int ta, const MapPlan &b, int tb) {
    const char *a0 = (const char *)a.base[ta];
    const char *a1 = a0 + 4 * (a.max_elem[ta] + 1);
    const char *b0 = (const char *)b.base[tb];
    const char *b1 = b0 + 4 * (b.max_elem[tb] + 1);
    if (a1 <= b0 || b1 <= a0)
        return true;
    if (a.rank != b.rank)
        return false;
    int64_t smin = 0;
    for (int d = 0; d < a.rank; ++d) {
        int64_t sa = a.stride[(size_t)ta * 4 + d], sb = b.stride[(size_t)tb * 4 + d];
        if (sa != sb)
            return false;
        if (sa > 0 && (smin == 0 || sa < smin))
            smin = sa;
    }
    if (smin <= 1)
        return false;
    for (int d = 0; d < a.rank; ++d)
        if (a.stride[(size_t)ta * 4 + d] % smin != 0)
            return false;
    int64_t diff = (int64_t)(b0 - a0);
    if (diff % 4 != 0)
        return false;
    return (diff / 4) % smin != 0;
}

Overlap classify_overlap(const MapPlan &in, const MapPlan &out) {
    // two `from` targets that can meet would race
    for (int a = 0; a < out.n_targets; ++a)
        for (int b = a + 1; b < out.n_targets; ++b)
            if (!disjoint_targets(out, a, out, b))
                return Overlap::OutputRace;
    for (int to = 0; to < out.n_targets; ++to)
        for (int ti = 0; ti < in.n_targets; ++ti) {
            if (disjoint_targets(in, ti, out, to))
                continue;
            // safe in one pass only as an element-for-element in-place update
            bool same = in.pointwise && in.base[ti] == out.base[to] && in.rank == out.rank;
            for (int d = 0; same && d < in.rank; ++d) {
                same = in.stride[(size_t)ti * 4 + d] == out.stride[(size_t)to * 4 + d] &&
                       in.start[d] == out.start[d] && in.step[d] == out.step[d] &&
                       in.count[d] == out.count[d] && out.omin[d] == 0 && out.omax[d] == 0;
            }
            if (!same)
                return Overlap::Snapshot;
        }
    return Overlap::None;
}

}  // namespace hpacml

// ---- convolutional models --------------------------------------------------

namespace hpacml {

hpacml_status validate_cnn(int32_t in_channels, int32_t height, int32_t width, int32_t n_layers,
                           const hpacml_layer *layers, CnnPlan *out) {
    if (!layers || n_layers < 1 || n_layers > HPACML_MAX_LAYERS)
        return HPACML_E_INVAL;
    if (in_channels < 1 || in_channels > HPACML_MAX_FEATURES || height < 1 || width < 1)
        return HPACML_E_INVAL;
    CnnPlan p;
    p.in_channels = in_channels;
    p.height = height;
    p.width = width;
    p.n_layers = n_layers;
    p.layers.assign(layers, layers + n_layers);
    int64_t h = height, w = width, c = in_channels;
    bool flat = false;
    p.shape.push_back({(int32_t)h, (int32_t)w, (int32_t)c});
    for (int l = 0; l < n_layers; ++l) {
        const hpacml_layer &y = layers[l];
        if (y.act != HPACML_ACT_IDENTITY && y.act != HPACML_ACT_RELU)
            return HPACML_E_INVAL;
        if (y.kind == HPACML_LAYER_LINEAR) {
            if (h * w * c > HPACML_MAX_CNN_WIDTH)
                return HPACML_E_UNSUPPORTED;
            c = y.out_channels;
            h = w = 1;
            flat = true;
        } else if (y.kind == HPACML_LAYER_CONV2D || y.kind == HPACML_LAYER_MAXPOOL2D) {
            if (flat)
                return HPACML_E_INVAL;
            if (y.kernel[0] < 1 || y.kernel[1] < 1 || y.stride[0] < 1 || y.stride[1] < 1)
                return HPACML_E_INVAL;
            const bool same = y.kind == HPACML_LAYER_CONV2D && y.padding == HPACML_PAD_SAME;
            if (y.kind == HPACML_LAYER_CONV2D) {
                if (y.padding != HPACML_PAD_SAME && y.padding != HPACML_PAD_VALID)
                    return HPACML_E_INVAL;
                if (same && (y.pad_mode < HPACML_PADMODE_ZEROS || y.pad_mode > HPACML_PADMODE_REPLICATE))
                    return HPACML_E_INVAL;
                if (y.kernel[0] > 64 || y.kernel[1] > 64)
                    return HPACML_E_UNSUPPORTED;
            }
            if (same) {
                if (y.stride[0] != 1 || y.stride[1] != 1)
                    return HPACML_E_INVAL;
            } else {
                if (y.kernel[0] > h || y.kernel[1] > w)
                    return HPACML_E_SHAPE;
                h = (h - y.kernel[0]) / y.stride[0] + 1;
                w = (w - y.kernel[1]) / y.stride[1] + 1;
            }
            if (y.kind == HPACML_LAYER_CONV2D)
                c = y.out_channels;
        } else {
            return HPACML_E_INVAL;
        }
        if (c < 1)
            return HPACML_E_INVAL;
        if (c > HPACML_MAX_CNN_WIDTH)
            return HPACML_E_UNSUPPORTED;
        p.shape.push_back({(int32_t)h, (int32_t)w, (int32_t)c});
    }
    for (const CnnShape &s : p.shape)
        p.max_elems = std::max(p.max_elems, (int64_t)s.h * s.w * s.c);
    if (out)
        *out = std::move(p);
    return HPACML_OK;
}

}  // namespace hpacml
