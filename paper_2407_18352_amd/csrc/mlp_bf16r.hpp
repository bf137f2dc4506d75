// bf16 fused region kernel with register-resident activations: gather -> MLP
// -> scatter for wide hidden layers (H in {256, 512}), bf16 operands with
// fp32 accumulation on v_mfma_f32_32x32x16_bf16.
//
// The surrogate runs per sweep point on the composed input tensor (Sec. IV-A
// composition, Sec. IV-B inference).  Each wave owns 64 points outright and
// keeps every activation of those points in its own registers (H x 64 bf16 =
// 64 KB at H = 512: 256 accumulation registers, read by the MFMA as its B
// operand), so no layer ever exchanges activations with another wave and no
// block-wide barrier separates the layers: the epilogue of one 32-feature
// block (bias, activation, bf16 rounding, and for the last hidden layer its
// share of the output layer) runs on the vector ALU while the matrix core
// works through the next block.  One wave per SIMD (512 registers).
//
// Every layer is computed transposed, H_out^T = W * H_in^T: A = 32 output
// features x 16 inputs of W (one 1 KB fragment), B = 16 inputs x 32 points of
// the activations (registers), C = 32 features x 32 points.  In the C layout
// lane l holds point l % 32 and, in register r, feature 8 (r / 4) + 4 (l / 32)
// + r % 4; registers 8t..8t+7, rounded to bf16, are directly the B operand of
// K-step 2j + t of the next layer when that layer's weight columns are
// permuted accordingly at pack time.  The first layer's bias rides in three
// bf16 columns of its zero-padded K; the hidden layers' biases (fp32) are
// added in the epilogue.
//
// The weights stream from L2 once per tile of 256 points (4 waves x 64) into
// a ring of 16 KB stages in LDS with direct global-to-LDS loads, each wave
// loading a quarter of every stage; all four waves read every fragment of it
// (each fragment feeds one MFMA per 32 points of the wave).  A stage is
// published by a wait for the wave's own loads and one barrier, taken a few
// fragments before the stage is needed.  The inputs of tile t + 2 are
// gathered during tile t through the `to` map, one direct load per feature
// and wave per stage, into a second LDS buffer, so their latency (window rows
// and planes that miss the caches) has a whole tile to pass.  The direct loads
// are issued as inline assembly the compiler does not see: seeing them, it
// would make every LDS read wait for all of them (it cannot tell one ring
// slot from another); their completion is this kernel's own count of
// vector-memory loads, and the barriers that publish their data are
// assembly with a memory clobber, so no LDS access moves across one.
#pragma once

#include <cfloat>
#include <cstddef>
#include <type_traits>

#include "kernels.hpp"

namespace hpacml {

namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));   // one fragment in registers

constexpr int kW = 4;                  // waves per block, one per SIMD
constexpr int kThreads = 64 * kW;
constexpr int kP = 64;                 // points per wave: two 32-point n-blocks
constexpr int kT = kW * kP;            // points per tile
constexpr int kFrag = 1024;            // one MFMA operand fragment: 64 lanes x 16 bytes
constexpr int kSF = 16;                // fragments per ring stage
constexpr int kStage = kSF * kFrag;    // 16 KB
constexpr int kPd = 7;                 // fragment reads in flight ahead of their use (7: 0.9% faster than 4)
constexpr int kR = 8;                  // fragments held in registers (> kPd, divides the layers' fragment counts)
constexpr int kSync = kSF - kPd - 2;   // fragment of a stage at which the next one is published
// after it, one direct load of the next ring stage per fragment, then the
// stage's gathers: the memory work of a stage goes out between matrix
// instructions instead of in one block after the barrier
static_assert(kSync + 5 < kSF, "four ring loads and the gathers fit after the barrier");
constexpr int kNS = 4;                 // ring stages in LDS
constexpr int kD = kNS - 1;            // stages loaded ahead
// scheduling-barrier mask: only VALU, SALU and transcendental instructions
// may be moved across (the matrix instructions and memory accesses keep
// their order)
constexpr int kSchedAluOnly = 0x2 | 0x4 | 0x400;

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// two fp32 -> packed bf16 pair (round to nearest even), one instruction
__device__ __forceinline__ uint32_t pack2(float a, float b) {
    const floatx2 v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// ReLU of an MFMA result that is rounded to bf16 next: one v_med3_f32(x, 0,
// FLT_MAX), which the compiler sees (so it keeps the wait states a vector
// ALU read of an MFMA result needs).  A NaN gives 0 (v_med3_f32 returns the
// minimum of the non-NaN operands then); +inf gives FLT_MAX, which rounds to
// bf16 +inf, so the bf16 result is that of max(x, 0) in every case.  (With an
// upper bound of +inf the compiler rewrites it as a maximum and quiets x
// first: two instructions.)
__device__ __forceinline__ float relu_to_bf16(float x) { return __builtin_amdgcn_fmed3f(x, 0.f, FLT_MAX); }

// registers 8t..8t+7 of a C fragment after ReLU, as a B fragment of the next
// layer (the bias is in the accumulator already)
__device__ __forceinline__ u32x4 to_b(const floatx16 &c, int t) {
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
        v[e] = relu_to_bf16(c[8 * t + e]);
    return u32x4{pack2(v[0], v[1]), pack2(v[2], v[3]), pack2(v[4], v[5]), pack2(v[6], v[7])};
}

// Keep an activation fragment in an accumulation register: the MFMA reads
// its B operand from there directly, which leaves the vector registers to
// everything the vector ALU touches (the activations of 64 points fill 256).
__device__ __forceinline__ u32x4 to_agpr(u32x4 v) {
    asm volatile("" : "+a"(v));
    return v;
}

// wait until at most N vector-memory loads of this wave are outstanding
template <int N>
__device__ __forceinline__ void vm_wait() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
// block barrier that no memory access (LDS included) moves across
__device__ __forceinline__ void block_barrier() { asm volatile("s_barrier" ::: "memory"); }

// direct global -> LDS loads (lane i's bytes land at lds + i * bytes; `lds`
// is wave-uniform); M0 is saved and restored around its use
__device__ __forceinline__ void dma16(const void *g, uint32_t lds) {
    uint32_t save;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %1, off\n\ts_mov_b32 m0, %0"
                 : "=&s"(save)
                 : "v"(g), "s"(lds)
                 : "memory");
}
__device__ __forceinline__ void dma4(const void *g, uint32_t lds) {
    uint32_t save;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\tglobal_load_lds_dword %1, off\n\ts_mov_b32 m0, %0"
                 : "=&s"(save)
                 : "v"(g), "s"(lds)
                 : "memory");
}

__device__ __forceinline__ uint32_t lds_addr(const void *p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)p;
}

// A map in one vector register: lane i holds 32-bit word i of its Map32, and
// a field is one v_readlane_b32 where it is used.  (Held by value, the maps'
// fields would sit in scalar registers for the whole kernel and spill.)
// `fresh()` hides the register's value from the compiler, so readings after
// it are made again rather than kept live from before.  Every dimension is
// resolved without branching on the rank: a map's unused dimensions have
// count 1, start 0, stride 0, extent 1 and no offsets, so they add nothing.
constexpr int kMapWords = (int)(sizeof(Map32) / 4);
static_assert(kMapWords <= 64, "one word per lane");
#define HPACML_MW(field) ((int)(offsetof(Map32, field) / 4))
struct LaneMap {
    int32_t v;
    __device__ void load(const Map32 &m, int lane) { v = ((const int32_t *)&m)[lane < kMapWords ? lane : 0]; }
    __device__ void fresh() { asm volatile("" : "+v"(v)); }
    __device__ int32_t word(int i) const { return __builtin_amdgcn_readlane(v, i); }
};

__device__ __forceinline__ Pt32 locate_lm(const LaneMap &m, int32_t b) {
    Pt32 r;
    uint32_t rem = (uint32_t)b;
    r.pe = 0;
#pragma unroll
    for (int d = HPACML_MAX_RANK - 1; d >= 0; --d) {
        const uint32_t magic = (uint32_t)m.word(HPACML_MW(magic) + d);
        const int32_t shift = m.word(HPACML_MW(shift) + d);
        const uint32_t q = (uint32_t)(((uint64_t)rem * magic) >> shift);
        const int32_t k = (int32_t)(rem - q * (uint32_t)m.word(HPACML_MW(count) + d));
        rem = q;
        const int32_t x = m.word(HPACML_MW(start) + d) + k * m.word(HPACML_MW(step) + d);
        r.p[d] = x;
        r.pe += x * m.word(HPACML_MW(stride) + d);
    }
    return r;
}

// A gather point: the element index of a sweep point and, per dimension,
// the smallest and largest offset that stay inside the arrays (-coordinate
// and extent - 1 - coordinate); unused dimensions give 0 and 0.
struct GPt {
    int32_t pe;
    int32_t lo[HPACML_MAX_RANK], hi[HPACML_MAX_RANK];
};

// Boundary correction of a windowed access (raw offsets raw8, signed bytes,
// wave-uniform) at gather point r: per dimension dl = clamp(offset, lo, hi)
// - offset (zero inside); clamp adds dl strides, periodic adds sign(dl)
// wraps (wmul = extent x stride, wlim = 1; one wrap suffices because the
// 32-bit plan keeps |offset| <= extent for periodic dimensions; clamp and
// unbounded dimensions have wmul = stride, wlim = INT32_MAX, and an
// unbounded dimension is never left).  Straight-line arithmetic, the same
// for every lane.
__device__ __forceinline__ int32_t gather_fix(const GPt &r, uint32_t raw8, const int32_t (&wmul)[HPACML_MAX_RANK],
                                              const int32_t (&wlim)[HPACML_MAX_RANK]) {
    uint32_t fix = 0;   // modulo 2^32: the corrected index itself fits in int32
#pragma unroll
    for (int d = 0; d < HPACML_MAX_RANK; ++d) {
        const int32_t o = (int32_t)(int8_t)(raw8 >> (8 * d));
        const int32_t dl = min(max(o, r.lo[d]), r.hi[d]) - o;
        fix += (uint32_t)min(max(dl, -wlim[d]), wlim[d]) * (uint32_t)wmul[d];
    }
    return (int32_t)fix;
}

// Boundary correction of the access with raw offsets raw8 (signed bytes,
// wave-uniform) at point r, added to the interior element index; the same
// straight-line arithmetic for every lane and every dimension, so that a
// gather carries no branch and the compiler can interleave it with the
// matrix instructions around it.  Per dimension, with q = coordinate +
// offset and dl = clamp(q, 0, n - 1) - q (zero inside the array): clamp adds
// dl strides; periodic adds sign(dl) * n strides, one wrap, which suffices
// because the 32-bit plan keeps |offset| <= extent for periodic dimensions.
// A dimension without a boundary mode is never left (the plan checks it),
// and an unused dimension has extent 1 and offset 0: both add zero.
__device__ __forceinline__ int32_t wrap_fix_lm(const LaneMap &m, const Pt32 &r, uint32_t raw8) {
    int32_t fix = 0;
#pragma unroll
    for (int d = 0; d < HPACML_MAX_RANK; ++d) {
        const int32_t off = (int32_t)(int8_t)(raw8 >> (8 * d));
        const int32_t n = m.word(HPACML_MW(extent) + d);
        const int32_t st = m.word(HPACML_MW(stride) + d);
        const bool per = m.word(HPACML_MW(bnd) + d) == HPACML_BND_PERIODIC;
        const int32_t lim = per ? 1 : INT32_MAX;
        const int32_t mul = per ? n * st : st;
        const int32_t q = r.p[d] + off;
        const int32_t dl = min(max(q, 0), n - 1) - q;
        fix += min(max(dl, -lim), lim) * mul;
    }
    return fix;
}

// compile-time loop: fn(std::integral_constant<int, i>) for i in [B, E)
template <int B, int E, typename Fn>
__device__ __forceinline__ void static_for(Fn &&fn) {
    if constexpr (B < E) {
        fn(std::integral_constant<int, B>{});
        static_for<B + 1, E>(fn);
    }
}

// Tile geometry and the weight stream of one tile.  The stream starts with
// layer 1 interleaved with the first hidden layer's m-block 0 (the fused
// region, padded to whole stages), in the order the kernel consumes them:
// for each layer-1 m-block j its K-steps, then (j >= 2) K-steps 2j - 4 and
// 2j - 3 of the hidden m-block 0; its last four K-steps close the region.
// The epilogues of layer 1 need more matrix instructions beside them than
// a first layer of one K-step, or one hidden m-block, provides; so hidden
// m-block 1 joins the region too (each of those K-steps is taken for m-block
// 0, then m-block 1) when the first layer has one K-step and another hidden
// layer follows, and when the first hidden layer is the last (its m-blocks'
// epilogues then feed the output layer in the m-block after the region).
// The hidden layers' other m-blocks follow, K-step by K-step.
constexpr bool fuse2(int ks1, int nh) { return (ks1 == 1 && nh >= 2) || nh == 1; }
constexpr int fused_mb(int ks1, int nh) { return fuse2(ks1, nh) ? 2 : 1; }
constexpr int fused_pos_l1(int ks1, int nh, int j, int s) {
    return j * ks1 + s + 2 * fused_mb(ks1, nh) * (j > 2 ? j - 2 : 0);
}
// hidden m-block m (< fused_mb) of the first hidden layer, K-step k
constexpr int fused_pos_h0(int ks1, int nh, int nmb, int k, int m) {
    const int fm = fused_mb(ks1, nh);
    return k < 2 * nmb - 4 ? fused_pos_l1(ks1, nh, k / 2 + 2, ks1 - 1) + 1 + fm * (k % 2) + m
                           : fused_pos_l1(ks1, nh, nmb - 1, ks1 - 1) + 1 + 2 * fm + fm * (k - (2 * nmb - 4)) + m;
}

template <int H, int NH, int KS1>
struct RGeo {
    static constexpr int NMB = H / 32;                    // 32-feature m-blocks
    static constexpr int KS = H / 16;                     // K-steps of a hidden layer
    static constexpr int L1F = NMB * KS1;                 // first-layer fragments
    static constexpr int HF = NMB * KS;                   // fragments of a hidden layer
    static constexpr bool F2 = fuse2(KS1, NH);            // hidden m-block 1 in the fused region
    static constexpr int FMB = fused_mb(KS1, NH);         // hidden m-blocks in the fused region
    static constexpr int FUSF = L1F + FMB * KS;           // fused region: layer 1 + those m-blocks
    static constexpr int FUS = (FUSF + kSF - 1) / kSF;    // ... in whole stages
    static constexpr int ST = FUS + (NH * HF - FMB * KS) / kSF; // stages per tile
    static constexpr int pos_l1(int j, int s) { return fused_pos_l1(KS1, NH, j, s); }
    static constexpr int pos_h0(int k, int m) { return fused_pos_h0(KS1, NH, NMB, k, m); }
    // m-block j of hidden layer l (l = 0: j >= FMB)
    static constexpr int pos_h(int l, int j) { return FUS * kSF - FMB * KS + (l * NMB + j) * KS; }
    static_assert(KS % kSF == 0, "hidden m-blocks are whole stages");
    static_assert(KS % kR == 0 && (FUS * kSF) % kR == 0, "fragment registers aligned with the layers");
    static_assert(NMB % 2 == 0 && NMB >= 4, "m-blocks go in pairs; the fused region needs four");
    static_assert(KS > 15, "an m-block's K-steps hold the previous epilogues (to K-step 15) and the output indices (10, 14)");
    static_assert(pos_h0(KS - 1, FMB - 1) == FUSF - 1, "the fused region is consumed in order");
    static_assert(pos_h0(0, 0) == pos_l1(2, KS1 - 1) + 1, "hidden K-steps follow layer-1 m-block 2");
    static_assert(pos_l1(3, 0) == pos_h0(1, FMB - 1) + 1, "layer-1 m-block 3 follows two hidden K-steps");
    static_assert(H != 512 || NH == 1, "512-wide activations fill the accumulation registers: one hidden layer");
};

template <int H, int NH, int KS1, int GPS, bool WIN>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
mlp_bf16r_kernel(Map32 in, Map32 out, FeatTable32 tin, FeatTable32 tout, BF16RPacked pk, int32_t n_tiles) {
    using G = RGeo<H, NH, KS1>;
    constexpr int NMB = G::NMB, KS = G::KS, ST = G::ST;
    extern __shared__ u32x4 smem[];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 5;
    const int col = lane & 31;
    const int F = in.n_features;
    // LDS: ring [kNS][16 KB] | X [2][kW][F][64] fp32 | W3 [NMB][2][2][8 rows]
    // x 16 B + a zero slot | hidden biases [NH][NMB][2][16] fp32
    char *lds = (char *)smem;
    const uint32_t lbase = lds_addr(smem);
    const int xoff = kNS * kStage;
    const int xbuf_bytes = kW * F * 256;
    const int xwave = w * F * 256;
    const int w3off = xoff + 2 * xbuf_bytes;
    const int zoff = w3off + NMB * 512;
    const int boff = zoff + 16;

    // the output-layer fragments (rows 0..7) and the hidden biases, staged
    // once by the block before any direct load is issued
    {
        u32x4 *w3l = (u32x4 *)(lds + w3off);
        const u32x4 *w3g = (const u32x4 *)pk.w3;
        for (int i = tid; i < NMB * 32; i += kThreads)
            w3l[i] = w3g[i];
        if (tid == 0)
            w3l[NMB * 32] = u32x4{0u, 0u, 0u, 0u};
        float *bl = (float *)(lds + boff);
        for (int i = tid; i < NH * NMB * 32; i += kThreads)
            bl[i] = pk.bias[i];
    }
    __syncthreads();

    // input feature table in registers: lane f holds feature f's pointer and
    // raw offsets; a wave-uniform feature is then three v_readlane_b32
    const int fl = lane < F ? lane : F - 1;
    const uint64_t tp = (uint64_t)(uintptr_t)tin.fptr[fl];
    const uint32_t t_lo = (uint32_t)tp, t_hi = (uint32_t)(tp >> 32), t_raw = tin.raw8[fl];
    // output table and biases the same way (the from map's outputs share
    // their raw offsets)
    const int ol = lane < 8 ? lane : 7;
    const uint64_t op = (uint64_t)(uintptr_t)tout.fptr[ol];
    const uint32_t o_lo = (uint32_t)op, o_hi = (uint32_t)(op >> 32);
    const uint32_t o_b = __builtin_bit_cast(uint32_t, pk.bias_out[ol]);
    const uint32_t o_raw = tout.raw8[0];
    const bool orelu = pk.act[pk.n_hidden + 1] == HPACML_ACT_RELU;
    LaneMap lin, lout;
    lin.load(in, lane);
    lout.load(out, lane);

    // XCD-aware tile order: blocks on one XCD take adjacent tiles
    const int nb = gridDim.x;
    const int lb = (nb % 8 == 0) ? (blockIdx.x % 8) * (nb / 8) + blockIdx.x / 8 : blockIdx.x;
    if (lb >= n_tiles)
        return;
    auto tile_of = [&](int it) { return lb + it * nb; };

    // gather of this wave's 64 points of a tile (lane = point), feature f
    // into X buffer xb; windowed maps (WIN) resolve boundaries per access
    // (per-dimension constants of the map: wrap multiplier and sign limit)
    int32_t wmul[HPACML_MAX_RANK], wlim[HPACML_MAX_RANK];
#pragma unroll
    for (int d = 0; d < HPACML_MAX_RANK; ++d) {
        const bool per = in.bnd[d] == HPACML_BND_PERIODIC;
        wmul[d] = per ? (int32_t)((uint32_t)in.extent[d] * (uint32_t)in.stride[d]) : in.stride[d];
        wlim[d] = per ? 1 : INT32_MAX;
    }
    auto gather_point = [&](int tile, GPt &gp) {
        int b = tile * kT + w * kP + lane;
        b = b < in.n_points ? b : in.n_points - 1;
        lin.fresh();
        const Pt32 pt = locate_lm(lin, b);
        gp.pe = pt.pe;
        if constexpr (WIN) {
#pragma unroll
            for (int d = 0; d < HPACML_MAX_RANK; ++d) {
                gp.lo[d] = -pt.p[d];
                gp.hi[d] = lin.word(HPACML_MW(extent) + d) - 1 - pt.p[d];
            }
        }
    };
    auto gather_one = [&](const GPt &gp, int f, int xb) {
        const uint32_t lo = __builtin_amdgcn_readlane(t_lo, f), hi = __builtin_amdgcn_readlane(t_hi, f);
        const float *base = (const float *)(uintptr_t)(((uint64_t)hi << 32) | lo);
        int32_t idx = gp.pe;
        if constexpr (WIN)
            idx += gather_fix(gp, __builtin_amdgcn_readlane(t_raw, f), wmul, wlim);
        dma4(base + idx, lbase + (uint32_t)(xoff + xb * xbuf_bytes + xwave + f * 256));
    };
    // ring stage k (global count) from the tile stream into slot k % kNS
    const char *wsrc = (const char *)pk.stream + (size_t)(4 * w) * kFrag + (size_t)lane * 16;
    // load i (of 4) of this wave's quarter of ring stage k
    auto ring_part = [&](int k, int i) {
        const int q = k % ST, slot = k % kNS;
        const char *src = wsrc + (size_t)q * kStage;
        const uint32_t dst = lbase + (uint32_t)(slot * kStage + 4 * w * kFrag);
        dma16(src + i * kFrag, dst + i * kFrag);
    };

    // ---- prologue: the first two tiles' inputs, the first kD stages
    {
        GPt gp;
        for (int i = 0; i < 2; ++i) {
            const int tt = tile_of(i) < n_tiles ? tile_of(i) : n_tiles - 1;
            gather_point(tt, gp);
            for (int f = 0; f < F; ++f)
                gather_one(gp, f, i);
        }
        for (int k = 0; k < kD; ++k)
            for (int i = 0; i < 4; ++i)
                ring_part(k, i);
        vm_wait<0>();
        block_barrier();
    }

    GPt gpt;                         // gather point of tile it + 2
    int gx = 0;                      // its X buffer
    int kb = 0;                      // global stage index of this tile's first stage
    const u32x4 *fr_lane = smem + lane;

    // Stage s of this tile, at fragment kSync: this wave's loads of stage
    // s + 1 have landed, then (barrier) every wave's, so stage s + 1 is
    // published.  The four loads of stage s + kD (into the slot of stage
    // s - 1, which every wave finished reading before the barrier) go out
    // at the next four fragments, the gathers of tile it + 2 at the fifth.
    // Between two barriers a wave issues GPS + 4 loads, so at the barrier at
    // most that many (the last stage's) may still be in flight.
    auto stage_work = [&](auto PS, int s) {
        constexpr int ps = decltype(PS)::value;
        if constexpr (ps == kSync) {
            vm_wait<(kD - 2) * (GPS + 4)>();
            block_barrier();
        } else if constexpr (ps > kSync && ps <= kSync + 4) {
            ring_part(kb + s + kD, ps - kSync - 1);
        } else if constexpr (ps == kSync + 5) {
#pragma unroll
            for (int i = 0; i < GPS; ++i) {
                const int f = s * GPS + i;
                gather_one(gpt, f < F ? f : F - 1, gx);
            }
        }
    };
    // the fragment pipeline: the read of the fragment at stream position
    // p + kPd is issued at position p (PC compile-time, pr a runtime multiple
    // of kSF), after the stage work of position p
    u32x4 a[kR];
    auto frag_ptr = [&](int p) { return fr_lane + ((kb + p / kSF) % kNS) * (kStage / 16) + (p % kSF) * (kFrag / 16); };
    auto fragment = [&](auto PC, int pr) -> bf16x8 {
        constexpr int pc = decltype(PC)::value;
        stage_work(std::integral_constant<int, pc % kSF>{}, (pc + pr) / kSF);
        a[(pc + kPd) % kR] = *frag_ptr(pc + pr + kPd);
        // keep the read kPd fragments ahead of its use: neither it nor the
        // matrix instructions may be moved across this point (the scheduler
        // would otherwise sink the read to just before its consumer and wait
        // for it there); vector and scalar ALU work still moves freely
        __builtin_amdgcn_sched_barrier(kSchedAluOnly);
        return as_bf16x8(a[pc % kR]);
    };
    // one K-step: the fragment at position PC (+ pr) times the B operands
    // b[0], b[1] into accumulators (c0, c1), which start from cinit when
    // FIRST (zero, or the layer's biases)
    auto kstep = [&](auto PC, int pr, const u32x4 (&b)[2], floatx16 &c0, floatx16 &c1, bool first,
                     const floatx16 &cinit) {
        const bf16x8 av = fragment(PC, pr);
        c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, as_bf16x8(b[0]), first ? cinit : c0, 0, 0, 0);
        c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, as_bf16x8(b[1]), first ? cinit : c1, 0, 0, 0);
    };
    // K loop of one m-block: K-step s at position PC0 + pr + s, B operands
    // hin[s]; mid(S) runs after K-step S (the previous m-block's epilogue,
    // spread over the loop)
    auto kloop = [&](auto PC0, int pr, auto NK, const u32x4 (*hin)[2], floatx16 &c0, floatx16 &c1,
                     const floatx16 &cinit, auto mid) {
        static_for<0, decltype(NK)::value>([&](auto S) {
            constexpr int s = decltype(S)::value;
            kstep(std::integral_constant<int, decltype(PC0)::value + s>{}, pr, hin[s], c0, c1, s == 0, cinit);
            mid(S);
        });
    };
    // biases of hidden layer l, m-block j, in the accumulator layout
    auto bias_of = [&](int l, int j) -> floatx16 {
        const floatx4 *bp = (const floatx4 *)(lds + boff + ((l * NMB + j) * 2 + g) * 64);
        floatx16 b;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const floatx4 v = bp[q];
            b[4 * q + 0] = v[0];
            b[4 * q + 1] = v[1];
            b[4 * q + 2] = v[2];
            b[4 * q + 3] = v[3];
        }
        return b;
    };
    // output-layer fragment t of m-block j (rows >= 8 read the zero slot)
    const int w3lane = (g * 8 + (col & 7)) * 16;
    auto wo_of = [&](int j, int t) -> bf16x8 {
        const int off = col < 8 ? w3off + (2 * j + t) * 256 + w3lane : zoff;
        return as_bf16x8(*(const u32x4 *)(lds + off));
    };

#pragma unroll
    for (int p = 0; p < kPd; ++p)
        a[p] = *frag_ptr(p);

    // ---- a tile's inputs (X buffer xbuf) as layer-1 B fragments; features
    //      F..F+2 carry the first-layer bias.  Rows below 16 (KS1 - 1) - 2
    //      (the fewest inputs of this K-step count) are inputs for every F;
    //      the others are read from a clamped row unconditionally and then
    //      masked without a branch: the input itself below F, 1 for the
    //      three bias columns, 0 above.  Piece (s, n) = K-step s, n-block n,
    //      in two parts: its LDS reads (xload), then the masking and packing
    //      (xfinish), issued apart so that waiting for the reads does not
    //      wait for the weight reads issued in between.
    constexpr int FMIN = 16 * (KS1 - 1) - 2;
    int32_t tb = 8 * g - F;                 // feature - F of element 0 of K-step 0 in this lane
    asm volatile("" : "+v"(tb));
    u32x4 xb[KS1][2];
    auto xload = [&](int xbuf, int s, int n, uint32_t (&v)[8]) {
        const float *xa = (const float *)(lds + xoff + xbuf * xbuf_bytes + xwave);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int f0 = 16 * s + e;
            if (16 * s + 8 + e < FMIN) {     // resolved at unrolling
                v[e] = __builtin_bit_cast(uint32_t, xa[(f0 + 8 * g) * 64 + 32 * n + col]);
            } else {
                const int32_t t = tb + f0;     // feature - F
                const int fc = t < 0 ? f0 + 8 * g : F - 1;
                v[e] = __builtin_bit_cast(uint32_t, xa[fc * 64 + 32 * n + col]);
            }
        }
    };
    auto xfinish = [&](int s, int n, uint32_t (&v)[8]) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            if (!(16 * s + 8 + e < FMIN)) {
                const int32_t t = tb + 16 * s + e;
                uint32_t x = v[e];
                asm volatile("" : "+v"(x));
                const uint32_t real = (uint32_t)(t >> 31);               // t < 0
                const uint32_t one = (uint32_t)((t - 3) >> 31) & 0x3F800000u;  // t < 3
                v[e] = (x & real) | (one & ~real);
            }
        }
        xb[s][n] = u32x4{pack2(__builtin_bit_cast(float, v[0]), __builtin_bit_cast(float, v[1])),
                         pack2(__builtin_bit_cast(float, v[2]), __builtin_bit_cast(float, v[3])),
                         pack2(__builtin_bit_cast(float, v[4]), __builtin_bit_cast(float, v[5])),
                         pack2(__builtin_bit_cast(float, v[6]), __builtin_bit_cast(float, v[7]))};
    };
    // the first tile's inputs (X buffer 0, landed in the prologue)
#pragma unroll
    for (int s = 0; s < KS1; ++s)
#pragma unroll
        for (int n = 0; n < 2; ++n) {
            uint32_t v[8];
            xload(0, s, n, v);
            xfinish(s, n, v);
        }

    u32x4 h[NH > 1 ? 2 : 1][KS][2];  // activations: B fragments [K-step][n-block]
    floatx16 acc[2][2];
    floatx16 hacc[2];                // m-block 0 of the first hidden layer
    floatx16 hacc1[G::F2 ? 2 : 1];   // ... and m-block 1 (F2)

    for (int it = 0; tile_of(it) < n_tiles; ++it) {
        const int tile = tile_of(it);
        {
            int tg = tile_of(it + 2);
            tg = tg < n_tiles ? tg : n_tiles - 1;
            gather_point(tg, gpt);
            gx = it & 1;
        }

        // ---- this tile's inputs are in xb (packed during the previous
        //      tile's last m-block, or by the prologue for the first tile)

        // ---- layer 1, fused with m-block 0 of the first hidden layer: for
        //      each m-block j of layer 1, its K-steps, then the epilogue of
        //      m-block j - 1 (activation, bf16 -> K-steps 2j - 2, 2j - 1 of
        //      the next layer), then K-steps 2j - 4, 2j - 3 of the hidden
        //      m-block 0, whose inputs the epilogue before made; the vector
        //      work of each epilogue runs beside ten matrix instructions, one
        //      quarter after each of its first four K-steps
        {
            // quarter q of the epilogue of layer-1 m-block j: K-step 2j + q / 2
            // of the next layer, n-block q % 2
            auto epi1 = [&](auto J, auto Q) {
                constexpr int j = decltype(J)::value, q = decltype(Q)::value;
                h[0][2 * j + q / 2][q % 2] = to_agpr(to_b(acc[j & 1][q % 2], q / 2));
            };
            const floatx16 zero = {};
            const floatx16 b00 = bias_of(0, 0);
            const floatx16 b01 = G::F2 ? bias_of(0, 1) : zero;
            auto h0 = [&](auto K) {
                constexpr int k = decltype(K)::value;
                kstep(std::integral_constant<int, G::pos_h0(k, 0)>{}, 0, h[0][k], hacc[0], hacc[1], k == 0, b00);
                if constexpr (G::F2)
                    kstep(std::integral_constant<int, G::pos_h0(k, 1)>{}, 0, h[0][k], hacc1[0],
                          hacc1[G::F2 ? 1 : 0], k == 0, b01);
            };
            static_for<0, NMB>([&](auto J) {
                constexpr int j = decltype(J)::value;
                constexpr int NK = KS1 + (j >= 2 ? 2 : 0);   // K-steps of this iteration
                using JP = std::integral_constant<int, (j >= 1 ? j - 1 : 0)>;
                static_for<0, NK>([&](auto I) {
                    constexpr int i = decltype(I)::value;
                    if constexpr (i < KS1)
                        kstep(std::integral_constant<int, G::pos_l1(j, i)>{}, 0, xb[i], acc[j & 1][0], acc[j & 1][1],
                              i == 0, zero);
                    else
                        h0(std::integral_constant<int, 2 * j - 4 + (i - KS1)>{});
                    if constexpr (j >= 1 && i < 4)
                        epi1(JP{}, I);
                });
                if constexpr (j >= 1)
                    static_for<(NK < 4 ? NK : 4), 4>([&](auto Q) { epi1(JP{}, Q); });
            });
            // the last epilogue, each half before the K-step that needs it
            using JL = std::integral_constant<int, NMB - 1>;
            static_for<0, 4>([&](auto Q) {
                epi1(JL{}, Q);
                h0(std::integral_constant<int, KS - 4 + decltype(Q)::value>{});
            });
            // padding fragments up to the stage boundary
            static_for<G::FUSF, G::FUS * kSF>([&](auto P) { (void)fragment(P, 0); });
        }

        // ---- hidden layers before the last: m-blocks unrolled (their
        //      activations land in statically indexed registers); the
        //      m-blocks of layer 0 in the fused region are done (their
        //      epilogues run in the first m-block here)
        static_for<0, NH - 1>([&](auto L) {
            constexpr int l = decltype(L)::value;
            const u32x4(*hin)[2] = h[l % 2];
            u32x4(*hout)[2] = h[(l + 1) % 2];
            // quarter q of the epilogue of m-block j (accumulators c)
            auto epih = [&](auto J, auto Q, floatx16 (&c)[2]) {
                constexpr int j = decltype(J)::value, q = decltype(Q)::value;
                hout[2 * j + q / 2][q % 2] = to_agpr(to_b(c[q % 2], q / 2));
            };
            static_for<(l == 0 ? G::FMB : 0), NMB>([&](auto J) {
                constexpr int j = decltype(J)::value;
                kloop(std::integral_constant<int, G::pos_h(l, j)>{}, 0, std::integral_constant<int, KS>{}, hin,
                      acc[j & 1][0], acc[j & 1][1], bias_of(l, j), [&](auto S) {
                          constexpr int s = decltype(S)::value;
                          // quarter q of the previous m-block's epilogue after
                          // K-step 1 + q KS / 4 (spread over the loop, so the
                          // vector work sits between matrix instructions)
                          constexpr int D = KS / 4;
                          if constexpr (j > 0 && s >= 1 && (s - 1) % D == 0 && (s - 1) / D < 4) {
                              using JP = std::integral_constant<int, (j > 0 ? j - 1 : 0)>;
                              using Q = std::integral_constant<int, (s - 1) / D>;
                              if constexpr (l == 0 && j == 1)
                                  epih(JP{}, Q{}, hacc);
                              else if constexpr (G::F2 && l == 0 && j == 2)
                                  epih(JP{}, Q{}, hacc1);
                              else
                                  epih(JP{}, Q{}, acc[(j - 1) & 1]);
                          }
                          // F2: the fused m-block 0's epilogue between m-block 1's quarters
                          if constexpr (G::F2 && l == 0 && j == 2 && s >= 1 + D / 2 && (s - 1 - D / 2) % D == 0 &&
                                        (s - 1 - D / 2) / D < 4)
                              epih(std::integral_constant<int, 0>{}, std::integral_constant<int, (s - 1 - D / 2) / D>{},
                                   hacc);
                      });
            });
            static_for<0, 4>([&](auto Q) { epih(std::integral_constant<int, NMB - 1>{}, Q, acc[(NMB - 1) & 1]); });
        });

        // ---- last hidden layer, streamed into the output layer: m-blocks in
        //      a loop of pairs; the epilogue of one (bias, activation, bf16,
        //      its share of the output layer) is spread over the next one's
        //      first K-steps
        {
            constexpr int l = NH - 1;
            const u32x4(*hin)[2] = h[l % 2];
            // stream position of m-block j is P0 + j KS (m-block 0 of a
            // single hidden layer was fused with layer 1)
            using P0 = std::integral_constant<int, G::pos_h(l, 0)>;
            using NKS = std::integral_constant<int, KS>;
            floatx16 y0 = {}, y1 = {};
            // part q of the epilogue of m-block j (accumulators c): K-step
            // t = q / 2 of the output layer for n-block q % 2
            auto epi_part = [&](auto Q, int j, floatx16 (&c)[2]) {
                constexpr int q = decltype(Q)::value, t = q >> 1;
                const bf16x8 wo = wo_of(j, t);
                if constexpr (q & 1) {
                    const u32x4 b1 = to_b(c[1], t);
                    y1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wo, as_bf16x8(b1), y1, 0, 0, 0);
                } else {
                    const u32x4 b0 = to_b(c[0], t);
                    y0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wo, as_bf16x8(b0), y0, 0, 0, 0);
                }
            };
            // element index of this lane's output point of n-block n (the
            // from map's boundary resolved), computed as vector filler
            // during m-block 1
            int32_t sidx[2];
            auto scatter_index = [&](int n) {
                const int b = tile * kT + w * kP + 32 * n + col;
                lout.fresh();
                const Pt32 pt = locate_lm(lout, b < out.n_points ? b : out.n_points - 1);
                lout.fresh();
                // a pointwise `from` map (no offsets: the usual case) never
                // leaves its arrays, so only a windowed one needs the fix-up
                sidx[n] = pt.pe + (o_raw != 0 ? wrap_fix_lm(lout, pt, o_raw) : 0);
            };
            // m-block j into accumulators cur; the epilogue of m-block j - 1
            // (accumulators prev) at K-steps 1, 3, 5, 7 (spreading them over the
            // loop, as the hidden layers before the last do, measured slower
            // here); extra(S) after K-step S
            auto mblock = [&](int j, floatx16 (&cur)[2], floatx16 (&prev)[2], bool first, auto extra) {
                kloop(P0{}, j * KS, NKS{}, hin, cur[0], cur[1], bias_of(l, j), [&](auto S) {
                    constexpr int s = decltype(S)::value;
                    if constexpr (s == 1 || s == 3 || s == 5 || s == 7) {
                        if (!first)
                            epi_part(std::integral_constant<int, (s >> 1)>{}, j - 1, prev);
                    }
                    extra(S);
                });
            };
            auto none = [](auto) {};
            auto indices = [&](auto S) {
                if constexpr (decltype(S)::value == 10)
                    scatter_index(0);
                if constexpr (decltype(S)::value == 14)
                    scatter_index(1);
            };
            // the first m-block pair after the fused region
            constexpr int J0 = NH == 1 && G::F2 ? 4 : 2;
            if constexpr (NH == 1 && G::F2) {
                // m-blocks 0 and 1 were computed in the fused region: m-block
                // 2 takes m-block 1's epilogue (K-steps 1-7) and m-block 0's
                // (K-steps 9-15), and the output indices
                auto two = [&](auto S) {
                    constexpr int s = decltype(S)::value;
                    if constexpr (s == 9 || s == 11 || s == 13 || s == 15)
                        epi_part(std::integral_constant<int, (s - 9) / 2>{}, 0, hacc);
                    indices(S);
                };
                mblock(2, acc[0], hacc1, false, two);
                mblock(3, acc[1], acc[0], false, none);
            } else if constexpr (NH == 1) {
                mblock(1, acc[1], hacc, false, indices);
            } else {
                mblock(0, acc[0], acc[1], true, none);
                mblock(1, acc[1], acc[0], false, indices);
            }
            for (int j = J0; j < NMB - 2; j += 2) {
                mblock(j, acc[0], acc[1], false, none);
                mblock(j + 1, acc[1], acc[0], false, none);
            }
            // the last m-block also packs the next tile's inputs (X buffer
            // (it + 1) & 1, gathered during the tile before this one): piece
            // p read after K-step 8 + p, finished after K-step 10 + p, in K-
            // steps that carry no other vector work
            uint32_t xv[2][8];
            const int nbuf = (it + 1) & 1;
            auto next_inputs = [&](auto S) {
                constexpr int s = decltype(S)::value, NP = 2 * KS1;
                if constexpr (s >= 10 && s < 10 + NP)
                    xfinish((s - 10) / 2, (s - 10) % 2, xv[(s - 10) % 2]);
                if constexpr (s >= 8 && s < 8 + NP)
                    xload(nbuf, (s - 8) / 2, (s - 8) % 2, xv[(s - 8) % 2]);
            };
            static_assert(KS >= 10 + 2 * KS1, "the next tile's inputs fit in the last m-block");
            mblock(NMB - 2, acc[0], acc[1], false, none);
            mblock(NMB - 1, acc[1], acc[0], false, next_inputs);
            static_for<0, 4>([&](auto Q) { epi_part(Q, NMB - 1, acc[1]); });

            // ---- scatter: y rows are outputs (row 4 g + r in register r < 4),
            //      lanes are points
#pragma unroll
            for (int n = 0; n < 2; ++n) {
                const floatx16 &y = n ? y1 : y0;
                const int b = tile * kT + w * kP + 32 * n + col;
                const int32_t idx = sidx[n];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int o = r + 4 * g;
                    if (o < pk.f_out && b < out.n_points) {
                        const uint32_t lo0 = __builtin_amdgcn_readlane(o_lo, r), lo1 = __builtin_amdgcn_readlane(o_lo, r + 4);
                        const uint32_t hi0 = __builtin_amdgcn_readlane(o_hi, r), hi1 = __builtin_amdgcn_readlane(o_hi, r + 4);
                        const float bo0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(o_b, r));
                        const float bo1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(o_b, r + 4));
                        float v = y[r] + (g ? bo1 : bo0);
                        if (orelu)
                            v = fmaxf(v, 0.f);
                        float *dst = (float *)(uintptr_t)(((uint64_t)(g ? hi1 : hi0) << 32) | (g ? lo1 : lo0));
                        stg(dst + idx, v);
                    }
                }
            }
        }
        kb += ST;
    }
    // every direct load has landed before the block's LDS is released
    vm_wait<0>();
}

// feature of the previous layer's output held at element e (lane half g) of
// K-step s of a B fragment built from C registers 8 (s % 2) .. + 7 of m-block
// s / 2
int b_feature(int s, int g, int e) { return 32 * (s / 2) + 16 * (s % 2) + 8 * (e / 4) + 4 * g + e % 4; }

int ring_stages(int H, int n_hidden, int ks1) {
    const int nmb = H / 32, ks = H / 16, fmb = fused_mb(ks1, n_hidden);
    const int fus = (nmb * ks1 + fmb * ks + kSF - 1) / kSF;
    return fus + (n_hidden * nmb * ks - fmb * ks) / kSF;
}

// first-layer K-steps and gathers per ring stage of a shape
int bf16r_ks1(int f_in) { return (f_in + 3 + 15) / 16; }
int bf16r_gps(int H, int n_hidden, int f_in) {
    const int st = ring_stages(H, n_hidden, bf16r_ks1(f_in));
    return (f_in + st - 1) / st;
}

// LDS of one block: ring, two input buffers, output fragments (+ a zero
// slot), hidden biases
size_t bf16r_lds_bytes(int H, int n_hidden, int f_in) {
    return (size_t)kNS * kStage + (size_t)2 * kW * f_in * 256 + (size_t)(H / 32) * 512 + 16 +
           (size_t)n_hidden * (H / 32) * 128;
}

template <int H, int NH, int KS1, int GPS>
hipError_t launch_r(const Map32 &in, const Map32 &out, const FeatTable32 &tin, const FeatTable32 &tout,
                    const BF16RPacked &pk, hipStream_t stream) {
    const int32_t n_tiles = (in.n_points + kT - 1) / kT;
    const size_t lds = bf16r_lds_bytes(H, NH, in.n_features);
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) == hipSuccess)
        (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    const int32_t grid = n_tiles < cus ? n_tiles : cus;
    // a map whose features all sit at the sweep point needs no boundary
    // resolution in its gathers
    bool win = false;
    for (int d = 0; d < HPACML_MAX_RANK; ++d)
        win = win || in.omin[d] != 0 || in.omax[d] != 0;
    auto kern = win ? mlp_bf16r_kernel<H, NH, KS1, GPS, true> : mlp_bf16r_kernel<H, NH, KS1, GPS, false>;
    hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kThreads), lds, stream, in, out, tin, tout, pk, n_tiles);
    return hipGetLastError();
}

}  // namespace

// launches of the 256-wide instantiations with NH hidden layers (each
// compiled in its own unit, so that they build in parallel)
template <int NH>
hipError_t launch_mlp_bf16r_h256(const Map32 &in, const Map32 &out, const FeatTable32 &tin, const FeatTable32 &tout,
                                 const BF16RPacked &pk, int gps, hipStream_t stream);

#define HPACML_BF16R_H256_UNIT(NH)                                                                              \
    template <>                                                                                                 \
    hipError_t launch_mlp_bf16r_h256<NH>(const Map32 &in, const Map32 &out, const FeatTable32 &tin,             \
                                         const FeatTable32 &tout, const BF16RPacked &pk, int gps,               \
                                         hipStream_t stream) {                                                  \
        if (pk.ks1 == 1)                                                                                        \
            return gps == 1 ? launch_r<256, NH, 1, 1>(in, out, tin, tout, pk, stream)                           \
                            : launch_r<256, NH, 1, 2>(in, out, tin, tout, pk, stream);                          \
        if (pk.ks1 == 2)                                                                                        \
            return gps == 1 ? launch_r<256, NH, 2, 1>(in, out, tin, tout, pk, stream)                           \
                            : launch_r<256, NH, 2, 2>(in, out, tin, tout, pk, stream);                          \
        return hipErrorInvalidValue;                                                                            \
    }

}  // namespace hpacml

