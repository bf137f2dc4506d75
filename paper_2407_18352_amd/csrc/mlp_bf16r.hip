// bf16 fused region kernel with register-resident activations: host side
// (shape support, weight-stream packing) and the 512-wide instantiations.
// The kernel itself is in mlp_bf16r.hpp.
#include "mlp_bf16r.hpp"

namespace hpacml {

bool bf16r_supported(int n_layers, const int32_t *dims, const int32_t *act, int compute) {
    if (compute != HPACML_BF16 || n_layers < 3)
        return false;
    const int H = dims[1], nh = n_layers - 2;
    if (!((H == 512 && nh == 1) || (H == 256 && nh <= 3)))
        return false;
    for (int l = 1; l < n_layers; ++l)
        if (dims[l] != H)
            return false;
    for (int l = 0; l + 1 < n_layers; ++l)
        if (act[l] != HPACML_ACT_RELU)
            return false;
    const int f_in = dims[0], ks1 = bf16r_ks1(f_in);
    if (dims[n_layers] > 8)
        return false;
    // instantiated shapes: 512 wide with 1-3 first-layer K-steps, 256 wide
    // with 1-3 hidden layers and 1-2 first-layer K-steps
    if (!((H == 512 && ks1 <= 3) || (H == 256 && ks1 <= 2)))
        return false;
    if (bf16r_lds_bytes(H, nh, f_in) > 160 * 1024)
        return false;
    return bf16r_gps(H, nh, f_in) <= 2;
}

// Stream of one tile: the fused region -- the first layer's fragments
// (column F..F+2 = the bias split in three bf16 terms) interleaved with the
// first hidden layer's m-block 0 (and 1), at fused_pos_l1 / fused_pos_h0 --
// padded to whole stages, then the hidden layers' other m-blocks in order
// (m-block j, K-step s, columns permuted to the B-fragment order).  A
// fragment is lane l = (i = l % 32, g = l / 32) x 8 elements: A[i][8 g + e].
void bf16r_pack(int n_layers, const int32_t *dims, const float *const *W, const float *const *b,
                std::vector<uint8_t> &buf, size_t *off_w3, size_t *off_bias, BF16RPacked *pk) {
    const int H = dims[1], F = dims[0], Fo = dims[n_layers];
    const int NMB = H / 32, KS = H / 16, nh = n_layers - 2;
    const int ks1 = bf16r_ks1(F);
    const int st = ring_stages(H, nh, ks1);
    const int fmb = fused_mb(ks1, nh);
    const int fus = (NMB * ks1 + fmb * KS + kSF - 1) / kSF;
    // stream position of K-step s of m-block j of hidden layer h
    auto pos_hidden = [&](int h, int j, int s) {
        return h == 0 && j < fmb ? fused_pos_h0(ks1, nh, NMB, s, j) : fus * kSF - fmb * KS + (h * NMB + j) * KS + s;
    };
    std::vector<uint16_t> stream((size_t)st * kSF * 64 * 8, 0);
    auto put = [&](int pos, int l, int e, uint16_t v) { stream[((size_t)pos * 64 + l) * 8 + e] = v; };
    for (int j = 0; j < NMB; ++j)
        for (int s = 0; s < ks1; ++s)
            for (int l = 0; l < 64; ++l)
                for (int e = 0; e < 8; ++e) {
                    const int o = 32 * j + l % 32, k = 16 * s + 8 * (l / 32) + e;
                    uint16_t v = 0;
                    if (k < F) {
                        v = bf16_rne_host(W[0][(size_t)o * F + k]);
                    } else if (k < F + 3) {
                        uint16_t t[3];
                        split_bias(b[0][o], t);
                        v = t[k - F];
                    }
                    put(fused_pos_l1(ks1, nh, j, s), l, e, v);
                }
    for (int h = 0; h < nh; ++h)
        for (int j = 0; j < NMB; ++j)
            for (int s = 0; s < KS; ++s)
                for (int l = 0; l < 64; ++l)
                    for (int e = 0; e < 8; ++e) {
                        const int o = 32 * j + l % 32;
                        const int k = b_feature(s, l / 32, e);
                        put(pos_hidden(h, j, s), l, e, bf16_rne_host(W[h + 1][(size_t)o * H + k]));
                    }
    // output layer: m-block j, K-step t, lane half g, row i < 8 (16 bytes each)
    std::vector<uint16_t> w3((size_t)NMB * 2 * 2 * 8 * 8, 0);
    for (int j = 0; j < NMB; ++j)
        for (int t = 0; t < 2; ++t)
            for (int g = 0; g < 2; ++g)
                for (int i = 0; i < 8; ++i)
                    for (int e = 0; e < 8; ++e) {
                        const int k = b_feature(2 * j + t, g, e);
                        w3[((((size_t)j * 2 + t) * 2 + g) * 8 + i) * 8 + e] =
                            i < Fo ? bf16_rne_host(W[n_layers - 1][(size_t)i * H + k]) : 0;
                    }
    std::vector<float> bias((size_t)nh * NMB * 2 * 16);
    for (int h = 0; h < nh; ++h)
        for (int j = 0; j < NMB; ++j)
            for (int g = 0; g < 2; ++g)
                for (int r = 0; r < 16; ++r)
                    bias[(((size_t)h * NMB + j) * 2 + g) * 16 + r] = b[h + 1][32 * j + 8 * (r / 4) + 4 * g + r % 4];
    buf.assign(stream.size() * 2 + w3.size() * 2 + bias.size() * 4, 0);
    std::memcpy(buf.data(), stream.data(), stream.size() * 2);
    *off_w3 = stream.size() * 2;
    std::memcpy(buf.data() + *off_w3, w3.data(), w3.size() * 2);
    *off_bias = *off_w3 + w3.size() * 2;
    std::memcpy(buf.data() + *off_bias, bias.data(), bias.size() * 4);
    pk->hid = H;
    pk->n_hidden = nh;
    pk->ks1 = ks1;
    pk->f_out = Fo;
    pk->stages = st;
    for (int i = 0; i < 16; ++i)
        pk->bias_out[i] = i < Fo ? b[n_layers - 1][i] : 0.f;
}

hipError_t launch_mlp_bf16r(const Map32 &in, const Map32 &out, const FeatTable32 &tin, const FeatTable32 &tout,
                            const BF16RPacked &pk, hipStream_t stream) {
    if (in.n_points == 0)
        return hipSuccess;
    const int gps = bf16r_gps(pk.hid, pk.n_hidden, in.n_features);
#define HPACML_R(H, NH, KS1)                                                                  \
    if (pk.hid == H && pk.n_hidden == NH && pk.ks1 == KS1)                                    \
        return gps == 1 ? launch_r<H, NH, KS1, 1>(in, out, tin, tout, pk, stream)         \
                        : launch_r<H, NH, KS1, 2>(in, out, tin, tout, pk, stream);
    HPACML_R(512, 1, 1)
    HPACML_R(512, 1, 2)
    HPACML_R(512, 1, 3)
#undef HPACML_R
    if (pk.hid == 256 && pk.n_hidden == 1)
        return launch_mlp_bf16r_h256<1>(in, out, tin, tout, pk, gps, stream);
    if (pk.hid == 256 && pk.n_hidden == 2)
        return launch_mlp_bf16r_h256<2>(in, out, tin, tout, pk, gps, stream);
    if (pk.hid == 256 && pk.n_hidden == 3)
        return launch_mlp_bf16r_h256<3>(in, out, tin, tout, pk, gps, stream);
    return hipErrorInvalidValue;
}

const char *bf16r_variant_name(const BF16RPacked &pk) {
    return pk.hid == 512 ? "mlp_bf16r_h512" : "mlp_bf16r_h256";
}

}  // namespace hpacml

