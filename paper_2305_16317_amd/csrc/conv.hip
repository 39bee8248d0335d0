// Per-pixel 4-layer stack (a stack of 1x1 convolutions) of the latent
// denoiser, fused into one kernel: k_conv_f32x3 for the fp32 network,
// k_conv_bf16 for the network with bf16 matmul operands.
//
// Both share one design.  Each wave owns a tile of 32 pixels of one sample
// and runs all four layers on it with the activations held in registers.
// Layers are computed transposed, out^T = W h^T: the MFMA's M dimension is the
// output feature and its N dimension the pixel.  Every 32x32 MFMA leaves
// D[i][j] in lane j + 32 ((i/4) % 2), register (i%4) + 4 (i/8), so the
// accumulator of output block nb holds, in lane l and register r, feature
// 32 nb + 8 (r/4) + 4 (l/32) + r%4 of pixel l%32.  On
// v_mfma_f32_32x32x16_bf16 and _f16 (A[i][k] in lane i + 32 (k/8), B[k][j] in
// lane j + 32 (k/8), element k%8 of 8 packed 16-bit values) accumulator
// registers 8 g2 .. 8 g2 + 7 of block b, activated, converted to 16 bits and
// packed, are exactly the B operand of k-step (b, g2) of the next layer
// (through an LDS exchange in k_conv_f32x3): lane half h then carries
// input features 32 b + 16 g2 + 8 (u/4) + 4 h + u%4, u = 0..7, and the host
// packs the weights with the same permutation of the reduction index.  No
// activation ever leaves the registers.
//
// Weights stream through LDS in slabs shared by a block's waves, double
// buffered: the next slab is copied global -> LDS by the gfx950 LDS-DMA path
// (global_load_lds_dwordx4, no registers involved) while the current one
// feeds the MFMAs.  The two buffers are separate LDS variables: with one
// array of two buffers the compiler cannot tell a read of one buffer from a
// copy into the other, and waits for every copy to land before the next read.
#include <cstring>
#include <utility>

#include "pd_internal.h"

namespace pd {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f16v __attribute__((ext_vector_type(16)));

// Compile-time loop: f(std::integral_constant<int, i>) for i in [0, N).  Every
// index into a register array must be a constant, or the array goes to
// scratch memory; #pragma unroll alone is not guaranteed on bodies this big.
template <class F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
    static_for_impl(f, std::make_integer_sequence<int, N>{});
}

__device__ __forceinline__ float silu(float v) {
    return v * __builtin_amdgcn_rcpf(1.0f + __expf(-v));
}

// Shift and bias vectors of the activations, staged in LDS: rows 0..NW-1 hold
// each wave's first-layer shift (b1 + e_n, plus Wc c on the guided branch)
// for the tile it is on, rows NW and NW+1 the biases b2 and b3.  Read from LDS,
// these values share the LDS counter with the weight fragments; read from
// global memory through a generic pointer they were flat loads, and every
// wait for a fragment also waited for them.
template <int NB, int NW>
struct ActVecs {
    static constexpr int W = 32 * NB;
    static constexpr int STRIDE = (W + 255) / 256 * 256;   // floats per row: whole 1 KB copies
    static constexpr int B2 = NW, B3 = NW + 1;              // bias rows
    static constexpr int ROWS = NW + 2;
    static constexpr int F4 = ROWS * STRIDE / 4;
};

// ---------------------------------------------------------------- bf16
// k_conv_bf16: every matmul operand is bf16 (round to nearest even);
// accumulation, bias, shift, SiLU and the guidance combination stay in fp32.
// Layer 1 pads K = C to 16 with zeros, layer 4 pads its C output rows to 32.
//
// A 32x32x16 bf16 MFMA and the SiLU of one accumulator register cost about
// the same issue time, so the work is arranged for the hardware to overlap
// them across waves: two blocks of 4 waves run per CU (two waves per SIMD, at
// most 256 registers each, one tile of 32 pixels per wave).  Each mid layer
// is streamed one output block at a time -- a slab holds that block's weights
// for every input -- and a wave activates the block as soon as its MFMAs end,
// so its SiLU work runs while the other block's wave on the SIMD is in its
// MFMAs.  Only one output block's accumulators are live at a time.
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));

constexpr int kBf16Waves = 4;

template <int NB, int C>
struct ConvLayoutBf16 {                          // units of 16 B (one lane's A operand)
    static constexpr int SL1 = NB * 64;          // layer 1: one k-step per output block
    static constexpr int SLM = 2 * NB * 64;      // one output block, every (input block, g2);
                                                 // layer 4 likewise (its C rows padded to 32)
    static constexpr int BUF = SL1 > SLM ? SL1 : SLM;
    static constexpr int TOTAL = SL1 + (2 * NB + 1) * SLM;
    // slab 0: layer 1; 1 + layer * NB + j: output block j of layer 2 or 3;
    // 1 + 2 NB: layer 4
    static constexpr __host__ __device__ int off(int i) { return i == 0 ? 0 : SL1 + (i - 1) * SLM; }
    static constexpr __host__ __device__ int size(int i) { return i == 0 ? SL1 : SLM; }
};

template <int NB, int C>
__global__ __launch_bounds__(kBf16Waves * 64) __attribute__((amdgpu_waves_per_eu(2, 2)))
void k_conv_bf16(ConvArgs a, RowSrc src, float* __restrict__ eps, int tiles_per_row) {
    using L = ConvLayoutBf16<NB, C>;
    constexpr int NW = kBf16Waves;
    using AV = ActVecs<NB, NW>;
    static_assert(C <= 8, "layer 1 holds at most 8 channels in one lane half");
    __shared__ bf8 lds_0[L::BUF];
    __shared__ bf8 lds_1[L::BUF];
    auto ldsb = [&](int buf) -> bf8* { return buf ? lds_1 : lds_0; };
    __shared__ f4 vec4[AV::F4];

    const int groups = src.active ? *src.active : src.max_groups;
    const int64_t ntiles = (int64_t)groups * src.group * tiles_per_row;
    const int64_t ngroups = (ntiles + NW - 1) / NW;
    if ((int64_t)blockIdx.x >= ngroups) return;              // uniform over the block

    const int tid = threadIdx.x, lane = tid & 63, half = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t P = a.P;

    // packed slab i -> LDS buffer `buf`, 1 KB per wave instruction
    auto dma = [&](int i, int buf) {
        const int nch = L::size(i) / 64;
        const char* gb = reinterpret_cast<const char*>(a.frags);
        uint32_t lo = (uint32_t)lane * 16u;
        asm volatile("" : "+s"(gb), "+v"(lo));
        bf8* ls = ldsb(buf);
        for (int c = wave; c < nch; c += NW) {
            const uint32_t ob = (uint32_t)(L::off(i) + c * 64) * 16u + lo;
            __builtin_amdgcn_global_load_lds(
                (const __attribute__((address_space(1))) void*)(gb + (size_t)ob),
                (__attribute__((address_space(3))) void*)(ls + c * 64), 16, 0, 0);
        }
    };
    auto land = [&]() {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
    };
    auto dma_shift = [&](int n, int br) {
        const float* row = (br == 0 ? a.shift_u : a.shift_c) + (int64_t)n * AV::W;
        float* dst = reinterpret_cast<float*>(vec4) + wave * AV::STRIDE;
        for (int c = 0; c < AV::STRIDE / 256; ++c) {
            int off = c * 256 + lane * 4;
            off = off <= AV::W - 4 ? off : AV::W - 4;
            __builtin_amdgcn_global_load_lds(
                (const __attribute__((address_space(1))) void*)(row + off),
                (__attribute__((address_space(3))) void*)(dst + c * 256), 16, 0, 0);
        }
    };
    // SiLU(acc + v) of block nb (v = LDS vector row vrow), rounded to bf16 and
    // packed as the block's two B operands
    auto act = [&](const f16v& c, int vrow, int nb, bf8 (&hb)[2]) {
        int o = vrow * (AV::STRIDE / 4);
        asm volatile("" : "+s"(o));
        static_for<4>([&](auto q4c) {
            constexpr int q4 = decltype(q4c)::value;
            const f4 sh = vec4[o + 8 * nb + 2 * q4 + half];
#pragma unroll
            for (int q = 0; q < 4; ++q) hb[q4 / 2][4 * (q4 % 2) + q] = (__bf16)silu(c[4 * q4 + q] + sh[q]);
        });
        // pinned here: left to itself the compiler sinks the activation to the
        // slab that first reads it, keeping 16 fp32 accumulators live in place
        // of 8 packed registers, and spills
        asm volatile("" : "+v"(hb[0]), "+v"(hb[1]));
    };
    struct Tile {
        int64_t row, px;
        bool active, pxok;
        const float* x;
        int n;
    };
    auto locate = [&](int64_t tg) -> Tile {
        Tile T;
        const int64_t tile = tg * NW + wave;
        T.active = tile < ntiles;
        const int64_t tt = T.active ? tile : ntiles - 1;
        T.row = tt / tiles_per_row;
        const int pt = (int)(tt % tiles_per_row);
        const int g = (int)(T.row / src.group), bb = (int)(T.row % src.group);
        const int64_t sl = src.slot ? __builtin_amdgcn_readfirstlane(src.slot[g]) : g;
        T.x = src.base + sl * src.slot_stride + (int64_t)bb * C * P;
        T.n = __builtin_amdgcn_readfirstlane(src.n[g]);
        T.px = (int64_t)pt * 32 + (lane & 31);
        T.pxok = T.px < P;
        return T;
    };
    // layer-1 input: channels 0..C-1 in lane half 0, zero padding elsewhere
    auto load_x = [&](const Tile& T) -> bf8 {
        bf8 xb;
        static_for<8>([&](auto uc) {
            constexpr int u = decltype(uc)::value;
            const float v = (half == 0 && u < C && T.pxok) ? T.x[u * P + T.px] : 0.f;
            xb[u] = (__bf16)v;
        });
        return xb;
    };
    const int nbranch = a.shift_c ? 2 : 1;

    Tile cur = locate(blockIdx.x);
    dma(0, 0);
    dma_shift(cur.n, 0);
    for (int i = tid; i < AV::W; i += NW * 64) {
        reinterpret_cast<float*>(vec4)[AV::B2 * AV::STRIDE + i] = a.b2[i];
        reinterpret_cast<float*>(vec4)[AV::B3 * AV::STRIDE + i] = a.b3[i];
    }
    land();
    bf8 xb = load_x(cur);

    for (int64_t tg = blockIdx.x; tg < ngroups; tg += gridDim.x) {
        const bool last_group = tg + gridDim.x >= ngroups;
        Tile nxt = locate(last_group ? tg : tg + gridDim.x);
        const bf8 xnx = load_x(nxt);

        float eu[4] = {0.f, 0.f, 0.f, 0.f};
        for (int br = 0; br < nbranch; ++br) {
            bf8 H[NB][2];

            // ---- layer 1 (slab 0, buffer 0): K = C padded to 16, activated
            // with this wave's shift (LDS row `wave`)
            dma(1, 1);
            static_for<NB>([&](auto jc) {
                constexpr int j = decltype(jc)::value;
                const f16v acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds_0[j * 64 + lane], xb, f16v{},
                                                                         0, 0, 0);
                act(acc, wave, j, H[j]);
            });

            // ---- layers 2 and 3: one slab (and one activation) per output block
            static_for<2>([&](auto lc) {
                constexpr int layer = decltype(lc)::value;
                bf8 Hn[NB][2];
                static_for<NB>([&](auto jc) {
                    constexpr int j = decltype(jc)::value;
                    constexpr int slab = 1 + layer * NB + j;
                    constexpr int buf = slab & 1;
                    land();                                      // this slab has landed
                    dma(slab + 1, buf ^ 1);                      // the next block or layer 4
                    f16v acc = f16v{};
                    static_for<NB>([&](auto bc) {
                        constexpr int b = decltype(bc)::value;
                        static_for<2>([&](auto g2c) {
                            constexpr int g2 = decltype(g2c)::value;
                            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ldsb(buf)[(b * 2 + g2) * 64 + lane],
                                                                          H[b][g2], acc, 0, 0, 0);
                        });
                    });
                    act(acc, layer == 0 ? AV::B2 : AV::B3, j, Hn[j]);
                });
                static_for<NB>([&](auto bc) {
                    constexpr int b = decltype(bc)::value;
                    H[b][0] = Hn[b][0];
                    H[b][1] = Hn[b][1];
                });
            });

            // ---- layer 4 (slab 1 + 2 NB, buffer 1)
            {
                constexpr int slab = 1 + 2 * NB;
                constexpr int buf = slab & 1;
                land();
                const bool more = br + 1 < nbranch || !last_group;
                if (more) {                                      // next pass's layer 1
                    dma(0, buf ^ 1);
                    if (br + 1 < nbranch) dma_shift(cur.n, br + 1);
                    else dma_shift(nxt.n, 0);
                }
                f16v o2[2] = {f16v{}, f16v{}};
                static_for<NB>([&](auto bc) {
                    constexpr int b = decltype(bc)::value;
                    static_for<2>([&](auto gc) {
                        constexpr int g2 = decltype(gc)::value;
                        o2[g2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ldsb(buf)[(b * 2 + g2) * 64 + lane],
                                                                         H[b][g2], o2[g2], 0, 0, 0);
                    });
                });
                const f16v o = o2[0] + o2[1];
                float* out = eps + cur.row * (int64_t)C * P;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int c = 4 * half + r;
                    if (c < C) {
                        const float v = o[r] + a.b4[c];
                        if (br == 0) {
                            eu[r] = v;
                            if (nbranch == 1 && cur.active && cur.pxok) out[c * P + cur.px] = v;
                        } else if (cur.active && cur.pxok) {
                            out[c * P + cur.px] = eu[r] + a.guidance * (v - eu[r]);
                        }
                    }
                }
                land();
            }
        }
        cur = nxt;
        xb = xnx;
    }
}

// ---------------------------------------------------------------- fp32
// k_conv_f32x3: the fp32 network with fp32-accurate products on
// v_mfma_f32_32x32x16_f16 for its two W x W layers.  Every fp32 operand is
// split exactly into a leading fp16 part and a scaled fp16 remainder:
// w = w0 + 2^-11 w1 with w0 the nearest fp16 to w and w1 the nearest fp16 to
// 2^11 (w - w0), so w is kept to 2^-22 |w|.  The three products
//   w0 (2^11 x0) + w0 x1 + w1 x0  =  2^11 (w0 x0 + w0 x1' + w1' x0)
// (x1' = 2^-11 x1, w1' = 2^-11 w1) go into one fp32 accumulator; the one left
// out, w1' x1', is about 2^-22 |w x|.  Each fp16 product is exact in fp32 and
// the sums are fp32.  The weights are split on the host into the two A
// operands w0 and w1.  The activations are split in registers into the three
// B operands 2^11 x0, x1 and x0, after a per-tile power-of-two scale s that
// puts the tile's largest input of the layer just below 2^4: 2^11 x0 then
// stays below 2^15, inside fp16's range, and values down to 2^-28 of the
// largest keep full precision.  The accumulator holds 2^11 s (W h), removed
// exactly by the next activation step.  The bound on the inputs comes from
// the pre-activation values, since |SiLU(u)| <= |u|.  A
// 32x32x16 fp16 MFMA does 16 times the multiply-adds of an fp32 one in the
// same time, so the three take 3/16 of the fp32 matrix-core time.
//
// Persistent blocks of 8 waves on 4 tiles: the two waves of a tile share a
// SIMD and split the output blocks of every layer between them (half 0 the
// first ceil(NB/2), half 1 the rest), so that one wave's SiLU and splitting
// run beside the other's MFMAs.  A tile's activations and a layer's
// accumulators would not fit one wave's 256 registers at two waves per SIMD;
// halved they do.  The owner of an input block activates it (fp32 SiLU) into
// an LDS exchange buffer one slab ahead, and both waves split it from there;
// at layer 4 each wave sums over its own input blocks and half 1 passes its
// partial sums to half 0 through the same buffer.
//
// Layer 1 (K = C) runs on fp32 MFMA (v_mfma_f32_32x32x2f32: A[i][k] in lane
// i + 32 k, B[k][j] in lane j + 32 k, the same accumulator layout); its slab
// holds, for output block nb and lane l, the C/2 values
// W1[32 nb + l%32][2 s + l/32].  Layers 2 and 3 run on the split products,
// with the weights split on the host: slab b holds input block b for every
// output block nb, fragment ((g2 NB + nb) 2 + part), one 16-B unit per lane.
// Layer 4 (C outputs) runs as fp32 fused multiply-adds on the VALU from W4
// in fp32 ([C][W], 5 KB at width 320): on the matrix core its C rows would be
// padded to 32.  LDS: two 40 KB slabs, two 16 KB exchange buffers and
// the activation vectors, 122,432 bytes at width 320.
typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float fl2 __attribute__((ext_vector_type(2)));

// 2^k for an integer |k| <= 126, built from its exponent field
__device__ __forceinline__ float pow2(int k) { return __builtin_bit_cast(float, (k + 127) << 23); }

template <int NB, int C>
struct ConvLayoutX3 {                            // units of 16 B
    static constexpr int KS1 = C / 2;            // layer-1 fp32 k-steps
    static constexpr int SL1 = (NB * 64 * KS1 / 4 + 63) / 64 * 64;
    static constexpr int SLM = 2 * NB * 2 * 64;
    static constexpr int SL4 = (C * 32 * NB / 4 + 63) / 64 * 64;   // layer 4: W4 in fp32, [C][W]
    static constexpr int BUF = SL1 > SLM ? SL1 : SLM;
    static constexpr int TOTAL = SL1 + 2 * NB * SLM + SL4;
    // slab 0: layer 1; 1 + layer * NB + b: input block b of layer 2 or 3;
    // 1 + 2 NB: layer 4
    static constexpr __host__ __device__ int off(int i) { return i == 0 ? 0 : SL1 + (i - 1) * SLM; }
    static constexpr __host__ __device__ int size(int i) {
        return i == 0 ? SL1 : i == 1 + 2 * NB ? SL4 : SLM;
    }
};

template <int NB, int C>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2)))
void k_conv_f32x3(ConvArgs a, RowSrc src, float* __restrict__ eps, int tiles_per_row) {
    using L = ConvLayoutX3<NB, C>;
    constexpr int NT = 4;                            // tiles per block, two waves each
    constexpr int NBH = (NB + 1) / 2;                // output blocks of half 0 (half 1: NB - NBH)
    constexpr int NPR = (NBH + 1) / 2;               // pairs of them
    constexpr int W = 32 * NB;
    static_assert(C % 2 == 0 && C <= 8, "layer 1 pairs channels; at most 8 channels");
    __shared__ bf8 lds_0[L::BUF];
    __shared__ bf8 lds_1[L::BUF];
    __shared__ f4 xch_0[NT * 4 * 64];                // one input block's activations per tile
    __shared__ f4 xch_1[NT * 4 * 64];
    __shared__ __attribute__((aligned(16))) float vec[(NT + 2) * W];   // shifts of the tiles, b2, b3
    __shared__ float s_max[2][NT][2];                // per layer, tile and half: largest |input|

    const int groups = src.active ? *src.active : src.max_groups;
    const int64_t ntiles = (int64_t)groups * src.group * tiles_per_row;
    const int64_t ngroups = (ntiles + NT - 1) / NT;
    if ((int64_t)blockIdx.x >= ngroups) return;              // uniform over the block

    const int tid = threadIdx.x, lane = tid & 63, half = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int tile = wave & (NT - 1);                // waves tile and tile + NT share a SIMD
    const int oh = wave >> 2;                        // output half
    const int64_t P = a.P;
    // does this wave own its j-th output block (half 1 has one fewer when NB is odd)
    auto own = [&](int j) { return NB % 2 == 0 || oh == 0 || j < NB - NBH; };

    auto ldsb = [&](int buf) -> bf8* { return buf ? lds_1 : lds_0; };
    auto xchb = [&](int buf) -> f4* { return (buf ? xch_1 : xch_0) + tile * 4 * 64; };
    auto dma = [&](int i, int buf) {                         // slab i -> buffer, 1 KB per wave op
        const int nch = L::size(i) / 64;
        const char* gb = reinterpret_cast<const char*>(a.frags);
        uint32_t lo = (uint32_t)lane * 16u;
        asm volatile("" : "+s"(gb), "+v"(lo));
        bf8* ls = ldsb(buf);
        for (int c = wave; c < nch; c += 2 * NT) {
            const uint32_t ob = (uint32_t)(L::off(i) + c * 64) * 16u + lo;
            __builtin_amdgcn_global_load_lds(
                (const __attribute__((address_space(1))) void*)(gb + (size_t)ob),
                (__attribute__((address_space(3))) void*)(ls + c * 64), 16, 0, 0);
        }
    };
    auto land = [&]() {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
    };
    // first-layer shift of this tile for the next pass (row n, branch br), by the tile's half-0 wave
    auto dma_shift = [&](int n, int br) {
        if (oh != 0) return;
        const float* row = (br == 0 ? a.shift_u : a.shift_c) + (int64_t)n * W;
        float* dst = vec + tile * W;
        for (int c = 0; c * 256 < W; ++c) {
            const int off = c * 256 + lane * 4;
            if (off < W)                                     // W is a multiple of 32
                __builtin_amdgcn_global_load_lds(
                    (const __attribute__((address_space(1))) void*)(row + off),
                    (__attribute__((address_space(3))) void*)(dst + c * 256), 16, 0, 0);
        }
    };
    // SiLU(cs acc + v) of output block nb, v = LDS vector row vrow, in fp32;
    // cs (a power of two) removes the scale the accumulator carries
    auto act = [&](const f16v& c, float cs, int vrow, int nb, f4 (&h)[4]) {
        const float* v = vec + vrow * W + 32 * nb + 4 * half;
        static_for<4>([&](auto q4c) {
            constexpr int q4 = decltype(q4c)::value;
            const f4 sh = *reinterpret_cast<const f4*>(v + 8 * q4);
#pragma unroll
            for (int q = 0; q < 4; ++q) h[q4][q] = silu(__builtin_fmaf(c[4 * q4 + q], cs, sh[q]));
        });
    };
    // largest |cs acc + v| over this wave's output blocks (the values act
    // takes the SiLU of), reduced over the wave
    auto in_max = [&](const f16v (&c)[NBH], float cs, int vrow) {
        float m = 0.f;
        static_for<NBH>([&](auto jc) {
            constexpr int j = decltype(jc)::value;
            if (own(j)) {
                const float* v = vec + vrow * W + 32 * (oh * NBH + j) + 4 * half;
                static_for<4>([&](auto q4c) {
                    constexpr int q4 = decltype(q4c)::value;
                    const f4 sh = *reinterpret_cast<const f4*>(v + 8 * q4);
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        m = __builtin_fmaxf(m, __builtin_fabsf(__builtin_fmaf(c[j][4 * q4 + q], cs, sh[q])));
                });
            }
        });
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) m = __builtin_fmaxf(m, __shfl_xor(m, o));
        return m;
    };
    // the fp16 parts 2^11 x0, x1 and x0 of half g2 of a block's activations,
    // scaled by sx: the B operands of its k-step g2
    auto split_g2 = [&](auto g2c, const f4 (&h)[4], float sx, h8 (&p)[2][3]) {
        constexpr int g2 = decltype(g2c)::value;
        static_for<2>([&](auto q4h) {
            constexpr int q4 = 2 * g2 + decltype(q4h)::value;
            static_for<2>([&](auto qc) {
                constexpr int q = 2 * decltype(qc)::value;
                constexpr int u = 4 * (q4 % 2) + q;
                const fl2 hv = fl2{h[q4][q], h[q4][q + 1]} * sx;        // exact
                const h2 x0 = __builtin_convertvector(hv, h2);
                const fl2 r = (hv - __builtin_convertvector(x0, fl2)) * 2048.f;   // exact
                const h2 x1 = __builtin_convertvector(r, h2);
                const h2 x0s = x0 * (_Float16)2048.f;                    // exact
                p[g2][0][u] = x0s[0]; p[g2][0][u + 1] = x0s[1];
                p[g2][1][u] = x1[0]; p[g2][1][u + 1] = x1[1];
                p[g2][2][u] = x0[0]; p[g2][2][u + 1] = x0[1];
            });
        });
    };
    auto mfma = [](const h8& w, const h8& x, const f16v& c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(w, x, c, 0, 0, 0);
    };
    // fragments w0, w1 of one output block against 2^11 x0, x1, x0
    auto mac3 = [&](const h8* fr, const h8 (&x)[3], f16v& acc) {
        const h8 w0 = fr[0], w1 = fr[64];
        acc = mfma(w0, x[0], acc);
        acc = mfma(w0, x[1], acc);
        acc = mfma(w1, x[2], acc);
    };
    auto mac3x2 = [&](const h8* fa, const h8* fb, const h8 (&x)[3], f16v& A, f16v& B) {
        const h8 a0 = fa[0], a1 = fa[64];
        const h8 b0 = fb[0], b1 = fb[64];
        A = mfma(a0, x[0], A);
        B = mfma(b0, x[0], B);
        A = mfma(a0, x[1], A);
        B = mfma(b0, x[1], B);
        A = mfma(a1, x[2], A);
        B = mfma(b1, x[2], B);
    };
    struct Tile {
        int64_t row, px;
        bool active, pxok;
        const float* x;
        int n;
    };
    auto locate = [&](int64_t tg) -> Tile {
        Tile T;
        const int64_t t = tg * NT + tile;
        T.active = t < ntiles;
        const int64_t tt = T.active ? t : ntiles - 1;       // idle waves redo the last tile
        T.row = tt / tiles_per_row;
        const int pt = (int)(tt % tiles_per_row);
        const int g = (int)(T.row / src.group), bb = (int)(T.row % src.group);
        const int64_t sl = src.slot ? __builtin_amdgcn_readfirstlane(src.slot[g]) : g;
        T.x = src.base + sl * src.slot_stride + (int64_t)bb * C * P;
        T.n = __builtin_amdgcn_readfirstlane(src.n[g]);
        T.px = (int64_t)pt * 32 + (lane & 31);
        T.pxok = T.px < P;
        return T;
    };
    const int nbranch = a.shift_c ? 2 : 1;

    Tile cur = locate(blockIdx.x);
    dma(0, 0);
    dma_shift(cur.n, 0);
    for (int i = tid; i < W; i += 2 * NT * 64) {
        vec[NT * W + i] = a.b2[i];
        vec[(NT + 1) * W + i] = a.b3[i];
    }
    land();
    float xin[L::KS1];
#pragma unroll
    for (int s = 0; s < L::KS1; ++s) xin[s] = cur.pxok ? cur.x[(2 * s + half) * P + cur.px] : 0.f;

    for (int64_t tg = blockIdx.x; tg < ngroups; tg += gridDim.x) {
        const bool last_group = tg + gridDim.x >= ngroups;
        Tile nxt = locate(last_group ? tg : tg + gridDim.x);
        float xnx[L::KS1];
#pragma unroll
        for (int s = 0; s < L::KS1; ++s) xnx[s] = nxt.pxok ? nxt.x[(2 * s + half) * P + nxt.px] : 0.f;

        float eu[C];
#pragma unroll
        for (int c = 0; c < C; ++c) eu[c] = 0.f;
        for (int br = 0; br < nbranch; ++br) {
            f16v acc[NBH];

            // ---- layer 1 (slab 0, buffer 0): this wave's output blocks on fp32 MFMA
            dma(1, 1);
            static_for<NBH>([&](auto jc) {
                constexpr int j = decltype(jc)::value;
                acc[j] = f16v{};
                if (own(j)) {
                    const float* f1 = reinterpret_cast<const float*>(lds_0) + ((oh * NBH + j) * 64 + lane) * L::KS1;
                    static_for<L::KS1>([&](auto sc) {
                        constexpr int s = decltype(sc)::value;
                        acc[j] = __builtin_amdgcn_mfma_f32_32x32x2f32(f1[s], xin[s], acc[j], 0, 0, 0);
                    });
                }
            });

            // ---- layers 2 and 3: one slab per input block; the block's owner
            // activates it into an exchange buffer one slab ahead.  cs is the
            // scale the accumulators carry (none after layer 1's fp32 MFMAs).
            float cs = 1.f;
            static_for<2>([&](auto lc) {
                constexpr int layer = decltype(lc)::value;
                const int vin = layer == 0 ? tile : NT;
                {
                    const float m = in_max(acc, cs, vin);
                    if (lane == 0) s_max[layer][tile][oh] = m;   // read after the next barrier
                }
                if (oh == 0) {
                    f4 h[4];
                    act(acc[0], cs, vin, 0, h);
                    f4* xd = xchb(0);
                    static_for<4>([&](auto q4c) { xd[decltype(q4c)::value * 64 + lane] = h[decltype(q4c)::value]; });
                }
                f16v nacc[NBH];
                static_for<NBH>([&](auto jc) { nacc[decltype(jc)::value] = f16v{}; });
                float sx = 1.f, cs_next = 1.f;
                static_for<NB>([&](auto bc) {
                    constexpr int b = decltype(bc)::value;
                    constexpr int slab = 1 + layer * NB + b;
                    constexpr int buf = slab & 1;
                    land();                                      // slab b and block b's activations are in
                    dma(slab + 1, buf ^ 1);
                    if constexpr (b == 0) {
                        // the tile's scale: its largest input m below 2^4, m 2^e < 2^(e+1)
                        const float m = __builtin_fmaxf(s_max[layer][tile][0], s_max[layer][tile][1]);
                        int e = 0;
                        if (m > 0.f && m <= 3.4028235e38f) {
                            const int be = (int)((__builtin_bit_cast(uint32_t, m) >> 23) & 0xff);
                            e = (be == 0 ? -126 : be - 127) - 3;
                            e = e < -100 ? -100 : (e > 120 ? 120 : e);   // 2^-e, 2^(e-11) normal
                        }
                        sx = pow2(-e);
                        cs_next = pow2(e - 11);
                    }
                    if constexpr (b + 1 < NB) {
                        constexpr int o = (b + 1) < NBH ? 0 : 1, jl = (b + 1) - o * NBH;
                        if (oh == o) {
                            f4 h[4];
                            act(acc[jl], cs, vin, b + 1, h);
                            f4* xd = xchb((b + 1) & 1);
                            static_for<4>([&](auto q4c) { xd[decltype(q4c)::value * 64 + lane] = h[decltype(q4c)::value]; });
                        }
                    }
                    const f4* xs = xchb(b & 1);
                    static_for<2>([&](auto g2c) {
                        constexpr int g2 = decltype(g2c)::value;
                        h8 X[2][3];
                        {
                            f4 h[4];
                            h[2 * g2] = xs[(2 * g2) * 64 + lane];
                            h[2 * g2 + 1] = xs[(2 * g2 + 1) * 64 + lane];
                            split_g2(g2c, h, sx, X);
                        }
                        static_for<NPR>([&](auto pc) {
                            constexpr int j = 2 * decltype(pc)::value;
                            const h8* fr = reinterpret_cast<const h8*>(ldsb(buf)) +
                                           ((g2 * NB + oh * NBH + j) * 2) * 64 + lane;
                            if constexpr (j + 1 < NBH) {
                                if (own(j + 1)) mac3x2(fr, fr + 2 * 64, X[g2], nacc[j], nacc[j + 1]);
                                else mac3(fr, X[g2], nacc[j]);
                            } else {
                                if (own(j)) mac3(fr, X[g2], nacc[j]);
                            }
                        });
                    });
                });
                static_for<NBH>([&](auto jc) { acc[decltype(jc)::value] = nacc[decltype(jc)::value]; });
                cs = cs_next;
            });

            // ---- layer 4 (slab 2NB+1, buffer 1: W4 in fp32): C outputs as fp32
            // dot products on the VALU, each half over its own input blocks, the
            // lane halves (the same pixel) added by a lane swap; half 1 hands its
            // sums to half 0
            {
                constexpr int slab = 1 + 2 * NB;
                constexpr int buf = slab & 1;
                constexpr int C4 = (C + 3) / 4;
                land();
                const bool more = br + 1 < nbranch || !last_group;
                if (more) {                                      // next pass's layer 1
                    dma(0, 0);
                    if (br + 1 < nbranch) dma_shift(cur.n, br + 1);
                    else dma_shift(nxt.n, 0);
                }
                const float* w4 = reinterpret_cast<const float*>(ldsb(buf));
                float part[4 * C4];
#pragma unroll
                for (int c = 0; c < 4 * C4; ++c) part[c] = 0.f;
                static_for<NBH>([&](auto jc) {
                    constexpr int j = decltype(jc)::value;
                    if (own(j)) {
                        f4 h[4];
                        act(acc[j], cs, NT + 1, oh * NBH + j, h);
                        static_for<4>([&](auto q4c) {
                            constexpr int q4 = decltype(q4c)::value;
                            const int f = 32 * (oh * NBH + j) + 8 * q4 + 4 * half;   // features f..f+3
                            static_for<C>([&](auto cc) {
                                constexpr int c = decltype(cc)::value;
                                const f4 w = *reinterpret_cast<const f4*>(w4 + c * W + f);
#pragma unroll
                                for (int q = 0; q < 4; ++q) part[c] = __builtin_fmaf(w[q], h[q4][q], part[c]);
                            });
                        });
                    }
                });
#pragma unroll
                for (int c = 0; c < C; ++c) part[c] += __shfl_xor(part[c], 32);
                f4* xp = xchb(0);
                if (oh == 1) {
#pragma unroll
                    for (int k = 0; k < C4; ++k)
                        xp[k * 64 + lane] = f4{part[4 * k], part[4 * k + 1], part[4 * k + 2], part[4 * k + 3]};
                }
                __syncthreads();
                if (oh == 0 && half == 0) {
                    float* out = eps + cur.row * (int64_t)C * P;
#pragma unroll
                    for (int k = 0; k < C4; ++k) {
                        const f4 o1 = xp[k * 64 + lane];
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            const int c = 4 * k + r;
                            if (c < C) {
                                const float v = (part[c] + o1[r]) + a.b4[c];
                                if (br == 0) {
                                    eu[c] = v;
                                    if (nbranch == 1 && cur.active && cur.pxok) out[c * P + cur.px] = v;
                                } else if (cur.active && cur.pxok) {
                                    out[c * P + cur.px] = eu[c] + a.guidance * (v - eu[c]);
                                }
                            }
                        }
                    }
                }
                land();                                          // slab 0 is in buffer 0 again
            }
        }
        cur = nxt;
#pragma unroll
        for (int s = 0; s < L::KS1; ++s) xin[s] = xnx[s];
    }
}

uint16_t to_bf16(float f) {                     // round to nearest even
    uint32_t u;
    std::memcpy(&u, &f, 4);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x40);
    const uint32_t lsb = (u >> 16) & 1u;
    return (uint16_t)((u + 0x7FFFu + lsb) >> 16);
}

template <int NB, int C>
void pack_bf16_t(const float* W1, const float* W2, const float* W3, const float* W4,
                 std::vector<uint8_t>& out) {
    using L = ConvLayoutBf16<NB, C>;
    constexpr int W = 32 * NB;
    out.assign((size_t)L::TOTAL * 16, 0);
    uint16_t* f = reinterpret_cast<uint16_t*>(out.data());     // 8 bf16 per unit
    auto unit = [&](int u) { return f + (size_t)u * 8; };
    for (int nb = 0; nb < NB; ++nb)
        for (int l = 0; l < 64; ++l)
            for (int u = 0; u < 8; ++u) {
                const int k = 8 * (l / 32) + u;
                unit(L::off(0) + nb * 64 + l)[u] =
                    k < C ? to_bf16(W1[(32 * nb + l % 32) * C + k]) : (uint16_t)0;
            }
    auto fin = [](int b, int g2, int l, int u) { return 32 * b + 16 * g2 + 8 * (u / 4) + 4 * (l / 32) + u % 4; };
    for (int layer = 0; layer < 2; ++layer) {
        const float* Wm = layer == 0 ? W2 : W3;
        for (int j = 0; j < NB; ++j)
            for (int b = 0; b < NB; ++b)
                for (int g2 = 0; g2 < 2; ++g2)
                    for (int l = 0; l < 64; ++l)
                        for (int u = 0; u < 8; ++u)
                            unit(L::off(1 + layer * NB + j) + (b * 2 + g2) * 64 + l)[u] =
                                to_bf16(Wm[(32 * j + l % 32) * W + fin(b, g2, l, u)]);
    }
    for (int b = 0; b < NB; ++b)
        for (int g2 = 0; g2 < 2; ++g2)
            for (int l = 0; l < 64; ++l)
                for (int u = 0; u < 8; ++u)
                    unit(L::off(1 + 2 * NB) + (b * 2 + g2) * 64 + l)[u] =
                        (l % 32 < C) ? to_bf16(W4[(l % 32) * W + fin(b, g2, l, u)]) : (uint16_t)0;
}

// The two A operands of an fp32 weight: w0, the nearest fp16 to w, and w1,
// the nearest fp16 to 2^11 (w - w0) (the difference is exact in fp32)
void split_f16(float w, uint16_t (&p)[2]) {
    if (!(w > -65504.f && w < 65504.f)) fail(PD_ERR_UNSUPPORTED, "fp32 conv weight outside fp16's range");
    const _Float16 w0 = (_Float16)w;
    const _Float16 w1 = (_Float16)((w - (float)w0) * 2048.f);
    std::memcpy(&p[0], &w0, 2);
    std::memcpy(&p[1], &w1, 2);
}

template <int NB, int C>
void pack_x3_t(const float* W1, const float* W2, const float* W3, const float* W4,
               std::vector<uint8_t>& out) {
    using L = ConvLayoutX3<NB, C>;
    constexpr int W = 32 * NB;
    out.assign((size_t)L::TOTAL * 16, 0);
    float* f = reinterpret_cast<float*>(out.data());            // layer 1: fp32 fragments
    for (int nb = 0; nb < NB; ++nb)
        for (int l = 0; l < 64; ++l)
            for (int s = 0; s < L::KS1; ++s)
                f[L::off(0) * 4 + (nb * 64 + l) * L::KS1 + s] = W1[(32 * nb + l % 32) * C + 2 * s + l / 32];
    uint16_t* h = reinterpret_cast<uint16_t*>(out.data());
    auto put = [&](int unit, int u, float w) {                  // part k -> k fragments on
        uint16_t p[2];
        split_f16(w, p);
        for (int k = 0; k < 2; ++k) h[((size_t)unit + (size_t)k * 64) * 8 + u] = p[k];
    };
    auto fin = [](int b, int g2, int l, int u) { return 32 * b + 16 * g2 + 8 * (u / 4) + 4 * (l / 32) + u % 4; };
    for (int layer = 0; layer < 2; ++layer) {
        const float* Wm = layer == 0 ? W2 : W3;
        for (int b = 0; b < NB; ++b)
            for (int g2 = 0; g2 < 2; ++g2)
                for (int nb = 0; nb < NB; ++nb)
                    for (int l = 0; l < 64; ++l)
                        for (int u = 0; u < 8; ++u)
                            put(L::off(1 + layer * NB + b) + ((g2 * NB + nb) * 2) * 64 + l, u,
                                Wm[(32 * nb + l % 32) * W + fin(b, g2, l, u)]);
    }
    float* f4w = f + (size_t)L::off(1 + 2 * NB) * 4;              // layer 4: fp32 [C][W]
    for (int c = 0; c < C; ++c)
        for (int k = 0; k < W; ++k) f4w[c * W + k] = W4[(size_t)c * W + k];
}

int device_cus();

template <int NB, int C>
void launch_bf16_t(const ConvArgs& a, const RowSrc& src, float* eps, hipStream_t s) {
    const int tiles_per_row = (int)((a.P + 31) / 32);
    const int64_t ntiles = (int64_t)src.max_groups * src.group * tiles_per_row;
    if (ntiles == 0) return;
    int64_t blocks = (ntiles + kBf16Waves - 1) / kBf16Waves;   // persistent: two blocks per CU
    if (blocks > 2 * device_cus()) blocks = 2 * device_cus();
    hipLaunchKernelGGL((k_conv_bf16<NB, C>), dim3((unsigned)blocks), dim3(kBf16Waves * 64), 0, s, a,
                       src, eps, tiles_per_row);
    PD_HIP(hipGetLastError());
}

int device_cus() {
    static int cus = 0;
    if (cus == 0) {
        int dev = 0;
        PD_HIP(hipGetDevice(&dev));
        PD_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
        if (cus <= 0) cus = 256;
    }
    return cus;
}

template <int NB, int C>
void launch_x3_t(const ConvArgs& a, const RowSrc& src, float* eps, hipStream_t s) {
    const int tiles_per_row = (int)((a.P + 31) / 32);
    const int64_t ntiles = (int64_t)src.max_groups * src.group * tiles_per_row;
    if (ntiles == 0) return;
    int64_t blocks = (ntiles + 3) / 4;                       // persistent: one block per CU
    if (blocks > device_cus()) blocks = device_cus();
    hipLaunchKernelGGL((k_conv_f32x3<NB, C>), dim3((unsigned)blocks), dim3(512), 0, s, a, src, eps,
                       tiles_per_row);
    PD_HIP(hipGetLastError());
}

// (blocks of 32 features, channels): widths 32, 64, 96, 128 and 320 over 4 channels
#define PD_CONV_SHAPES(X) X(1, 4) X(2, 4) X(3, 4) X(4, 4) X(10, 4)

}  // namespace

bool conv_supported(int C, int width, bool bf16) {
#define X(nb, c) if (C == c && width == 32 * nb) return true;
    PD_CONV_SHAPES(X)
#undef X
    (void)bf16;
    return false;
}

size_t conv_frag_bytes(int C, int width, bool bf16) {
#define X(nb, c)                                                                      \
    if (C == c && width == 32 * nb)                                                   \
        return bf16 ? (size_t)ConvLayoutBf16<nb, c>::TOTAL * 16 : (size_t)ConvLayoutX3<nb, c>::TOTAL * 16;
    PD_CONV_SHAPES(X)
#undef X
    return 0;
}

void conv_pack_weights(int C, int width, bool bf16, const float* W1, const float* W2,
                       const float* W3, const float* W4, std::vector<uint8_t>& out) {
#define X(nb, c)                                                  \
    if (C == c && width == 32 * nb) {                             \
        if (bf16)                                                 \
            pack_bf16_t<nb, c>(W1, W2, W3, W4, out);              \
        else                                                      \
            pack_x3_t<nb, c>(W1, W2, W3, W4, out);                \
        return;                                                   \
    }
    PD_CONV_SHAPES(X)
#undef X
    fail(PD_ERR_UNSUPPORTED, "conv1x1: unsupported channel count / width");
}

void launch_conv1x1(const ConvArgs& a, const RowSrc& src, float* eps, hipStream_t s) {
#define X(nb, c)                                                   \
    if (a.C == c && a.width == 32 * nb) {                          \
        if (a.bf16)                                                \
            launch_bf16_t<nb, c>(a, src, eps, s);                  \
        else                                                       \
            launch_x3_t<nb, c>(a, src, eps, s);                    \
        return;                                                    \
    }
    PD_CONV_SHAPES(X)
#undef X
    fail(PD_ERR_UNSUPPORTED, "conv1x1: unsupported channel count / width");
}

}  // namespace pd
