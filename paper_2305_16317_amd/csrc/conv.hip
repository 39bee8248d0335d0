// Per-pixel 4-layer stack (a stack of 1x1 convolutions) of the latent
// denoiser, fused into one kernel: k_conv_f32s for the fp32 network,
// k_conv_bf16 for the network with bf16 matmul operands.
//
// Both run all four layers of a pixel tile inside the waves that own it, with
// the activations in registers.  Layers are computed transposed,
// out^T = W h^T: the MFMA's M dimension is the output feature and its N
// dimension the pixel, so a layer's accumulators, activated and converted to
// 16 bits, are the next layer's B operands once the host packs the weights
// with the matching permutation of the reduction index (each kernel's layout
// comment gives it).  No activation leaves the registers.
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

// SiLU(u) from t = kNegLog2e u: e = 2^t = e^-u and SiLU(u) = u / (1 + e) =
// t / ((1 + e) kNegLog2e), the constant cancelling exactly (the same float in
// t and in the fused multiply-add)
__device__ __forceinline__ float silu_t(float t) {
    return t * __builtin_amdgcn_rcpf(__builtin_fmaf(__builtin_amdgcn_exp2f(t), kNegLog2e, kNegLog2e));
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
    // SiLU(acc + v) of block nb (v = LDS vector row vrow, held times
    // kNegLog2e), rounded to bf16 and packed as the block's two B operands
    auto act = [&](const f16v& c, int vrow, int nb, bf8 (&hb)[2]) {
        int o = vrow * (AV::STRIDE / 4);
        asm volatile("" : "+s"(o));
        static_for<4>([&](auto q4c) {
            constexpr int q4 = decltype(q4c)::value;
            const f4 sh = vec4[o + 8 * nb + 2 * q4 + half];
#pragma unroll
            for (int q = 0; q < 4; ++q)
                hb[q4 / 2][4 * (q4 % 2) + q] = (__bf16)silu_t(__builtin_fmaf(c[4 * q4 + q], kNegLog2e, sh[q]));
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
        T.n = __builtin_amdgcn_readfirstlane(row_timestep(src, g));
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
typedef _Float16 h8 __attribute__((ext_vector_type(8)));

// Largest value over the wave, the same in every lane: DPP steps build the
// maximum of each 16-lane row in every lane of it (pairs, quads, half rows,
// rows), two row broadcasts carry it into the last row, and lane 63 is read.
// Maximum is exact, so any order of the steps gives the same value.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_max_step(float m) {
    // lanes outside ROW_MASK keep their own value
    const int v = __builtin_bit_cast(int, m);
    return __builtin_fmaxf(m, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(v, v, CTRL, ROW_MASK, 0xf, false)));
}
__device__ __forceinline__ float wave_max_dpp(float m) {
    m = dpp_max_step<0xb1, 0xf>(m);    // quad_perm [1,0,3,2]
    m = dpp_max_step<0x4e, 0xf>(m);    // quad_perm [2,3,0,1]
    m = dpp_max_step<0x141, 0xf>(m);   // row_half_mirror
    m = dpp_max_step<0x140, 0xf>(m);   // row_mirror
    m = dpp_max_step<0x142, 0xa>(m);   // row_bcast:15 into rows 1 and 3
    m = dpp_max_step<0x143, 0xc>(m);   // row_bcast:31 into rows 2 and 3
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, m), 63));
}

// 2^k for an integer |k| <= 126, built from its exponent field
__device__ __forceinline__ float pow2(int k) { return __builtin_bit_cast(float, (k + 127) << 23); }

// ---------------------------------------------------------------- fp32, 16-pixel tiles
// k_conv_f32s: the fp32 network with the same split products, one wave per
// tile of 16 pixels, every output feature of every layer in that wave.  Each
// wave is self-contained: its activations never leave its registers, so no
// two waves exchange data and the only synchronisation is the weight stream.
// Eight waves (two per SIMD, on different tiles) share each streamed slab.
//
// v_mfma_f32_16x16x32_f16 (A[i][k] in lane i + 16 (k/8), B[k][j] in lane
// j + 16 (k/8), element k%8 of 8 packed halves; D[i][j] in lane j + 16 (i/4),
// register i%4): the accumulator of output block o (16 features) holds, in
// lane l and register r, feature 16 o + 4 (l/16) + r of pixel l%16.
// Registers 0..3 of blocks 2c and 2c + 1, activated and split, are the B
// operands of reduction chunk c (32 inputs) of the next layer: lane group
// g = l/16 carries inputs 32 c + 16 (u/4) + 4 g + u%4, u = 0..7, and the host
// packs the weights with the same permutation.  Layer 1 (K = C = 4) is one
// v_mfma_f32_16x16x4f32 per output block (A[i][k], B[k][j] in lanes i + 16 k,
// j + 16 k; the same accumulator layout); layer 4 (C outputs) is one output
// block whose rows past C are zero, on the split products like the mid
// layers.
//
// Split products: the weights w = w0 + 2^-11 w1 as before.  The activation
// h = SiLU(u) of a layer's input enters scaled, hs = S h with S = 2^(11-e) a
// power of two per tile and layer that puts the tile's largest input below
// 2^15 (e from its largest |t|, below): x0s = fp16(hs), x1 = fp16(hs - x0s) and
// x0 = x0s 2^-11, so that w0 x0s + w0 x1 + w1 x0 = S (w h) to about 2^-22
// |w h|, every fp16 product exact in fp32.  A pre-activation u is carried as
// t = kNegLog2e u, the base-2 argument of e^-u, so that no multiply precedes
// the exponential: the epilogue forms t = acc (kNegLog2e / S) + kNegLog2e b
// in one fused multiply-add (the scaling exact, the bias row pre-multiplied).
// SiLU and the split fuse: with e = 2^t and r = 1 / ((1 + e) kNegLog2e / S)
// (one fused multiply-add for the product, the scale an exact power of two),
// t r = S u / (1 + e) = hs.  x0s = fp16(fl(t r)) (v_cvt_pk_f16_f32, two values
// per instruction, nearest even), the remainder t r - x0s is formed exactly and
// rounded once to fp32 (v_fma_mix_f32, the fp16 operand read in place), and
// x1 = fp16 of it; both fp16 roundings are the half-rate conversions, not the
// quarter-rate fp16-result v_fma_mix.  The next layer's accumulator holds
// S (W h).
typedef uint32_t u4v __attribute__((ext_vector_type(4)));

template <int NB, int C>
struct LayoutS {                                  // units of 16 B (one lane's operand)
    static constexpr int NO = 2 * NB;             // 16-feature output blocks of a W-wide layer
    static constexpr int KC = NB;                 // 32-input reduction chunks
    static constexpr int L1 = (NO * 16 + 63) / 64 * 64;   // layer 1: one fp32 per lane per block
    static constexpr int L4 = KC * 2 * 64;        // layer 4: parts w0, w1 per chunk
    static constexpr int RES = L1 + L4;           // resident in LDS for the whole kernel
    static constexpr int SLAB = NO * 2 * 64;      // one chunk of a mid layer: every block, both parts
    static constexpr int TOTAL = RES + 2 * KC * SLAB;
    static constexpr __host__ __device__ int mid(int layer, int c) { return RES + (layer * KC + c) * SLAB; }
};

// SiLU and split of 8 inputs (registers 0..3 of two output blocks): the B
// operands x0s, x1, x0 of one reduction chunk.  The inputs arrive as
// t = kNegLog2e u (u the pre-activation) and c = kNegLog2e / S.  The work comes
// in four pieces of two inputs (q = 0..3, packed register q of each operand)
// and a final one (x0), so that it can be spread between MFMA groups.
struct SplitB {
    u4v p0, p1, p2;
};
// stage 1 of two inputs: e = 2^t = e^-u and r = 1 / ((1 + e) c); the fused
// multiply-add forms (1 + e) c with one rounding, and t r = S u / (1 + e) =
// S SiLU(u) since the same float constant kNegLog2e is in t and in c
struct SplitR { float r0, r1; };
__device__ __forceinline__ SplitR silu_r(const float v0, const float v1, float c) {
    return {__builtin_amdgcn_rcpf(__builtin_fmaf(__builtin_amdgcn_exp2f(v0), c, c)),
            __builtin_amdgcn_rcpf(__builtin_fmaf(__builtin_amdgcn_exp2f(v1), c, c))};
}
// stage 2: x0s = fp16(fl(t r)) and x1 = fp16(t r - x0s), two halves each
__device__ __forceinline__ void split_round(const float v0, const float v1, const SplitR& r,
                                            uint32_t& x0s, uint32_t& x1) {
    const float h0 = v0 * r.r0, h1 = v1 * r.r1;
    uint32_t a, b;
    float d0, d1;
    asm("v_cvt_pk_f16_f32 %0, %1, %2" : "=v"(a) : "v"(h0), "v"(h1));
    asm("v_fma_mix_f32 %0, %1, %2, -%3 op_sel_hi:[0,0,1]" : "=v"(d0) : "v"(v0), "v"(r.r0), "v"(a));
    asm("v_fma_mix_f32 %0, %1, %2, -%3 op_sel:[0,0,1] op_sel_hi:[0,0,1]" : "=v"(d1) : "v"(v1), "v"(r.r1), "v"(a));
    asm("v_cvt_pk_f16_f32 %0, %1, %2" : "=v"(b) : "v"(d0), "v"(d1));
    x0s = a;
    x1 = b;
}
__device__ __forceinline__ void silu_split_q(const float v0, const float v1, float c,
                                             uint32_t& x0s, uint32_t& x1) {
    split_round(v0, v1, silu_r(v0, v1, c), x0s, x1);
}
__device__ __forceinline__ float f4_at(const f4& ua, const f4& ub, int i) { return i < 4 ? ua[i] : ub[i - 4]; }
__device__ __forceinline__ void silu_split_piece(int q, const f4& ua, const f4& ub, float c, SplitB& s) {
    if (q < 4) {
        uint32_t a, b;
        silu_split_q(f4_at(ua, ub, 2 * q), f4_at(ua, ub, 2 * q + 1), c, a, b);
        s.p0[q] = a;
        s.p1[q] = b;
    } else {                                         // x0 = x0s 2^-11
        s.p2 = __builtin_bit_cast(u4v, __builtin_bit_cast(h8, s.p0) * (_Float16)0.00048828125f);
    }
}
// the same work in nine steps of about six vector instructions, to spread
// between MFMA groups: step 2q is stage 1 of inputs 2q, 2q + 1, step 2q + 1
// their stage 2, step 8 forms x0
__device__ __forceinline__ void silu_split_step(int k, const f4& ua, const f4& ub, float c, SplitB& s, SplitR& st) {
    if (k < 8) {
        const int q = k >> 1;
        const float v0 = f4_at(ua, ub, 2 * q), v1 = f4_at(ua, ub, 2 * q + 1);
        if ((k & 1) == 0) {
            st = silu_r(v0, v1, c);
        } else {
            uint32_t a, b;
            split_round(v0, v1, st, a, b);
            s.p0[q] = a;
            s.p1[q] = b;
        }
    } else {                                         // x0 = x0s 2^-11
        s.p2 = __builtin_bit_cast(u4v, __builtin_bit_cast(h8, s.p0) * (_Float16)0.00048828125f);
    }
}
__device__ __forceinline__ SplitB silu_split(const f4& ua, const f4& ub, float c) {
    SplitB s;
#pragma unroll
    for (int q = 0; q < 5; ++q) silu_split_piece(q, ua, ub, c, s);
    return s;
}

// One LDS-DMA copy, 16 B per lane from gbase + voff to the LDS address lds +
// 16 lane (global_load_lds_dwordx4, M0 = lds), issued as inline assembly: the
// compiler's wait-count pass does not see it, so it keeps counting the
// kernel's own LDS reads precisely (with an LDS-DMA in flight it would wait
// for every outstanding LDS read before each use).  Callers wait for these
// copies explicitly (s_waitcnt vmcnt(0)) before any wave reads their data.
// The base address is uniform over the wave by construction; readfirstlane
// puts it in scalar registers, as the instruction needs.
__device__ __forceinline__ uint64_t uniform_addr(const void* p) {
    const uint64_t v = (uint64_t)(uintptr_t)p;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ void dma16(const void* gbase, uint32_t voff, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %2\n\t"
                 "global_load_lds_dwordx4 %0, %1"
                 :
                 : "v"(voff), "s"(uniform_addr(gbase)), "s"(__builtin_amdgcn_readfirstlane(lds))
                 : "memory", "m0");
}
__device__ __forceinline__ void dma4(const void* gbase, uint32_t voff, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %2\n\t"
                 "global_load_lds_dword %0, %1"
                 :
                 : "v"(voff), "s"(uniform_addr(gbase)), "s"(__builtin_amdgcn_readfirstlane(lds))
                 : "memory", "m0");
}
template <class T>
__device__ __forceinline__ uint32_t lds_addr(T* p) {
    return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) T*)p;
}

template <int NB, int C, bool GUIDED>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2)))
void k_conv_f32s(ConvArgs a, RowSrc src, float* __restrict__ eps, int tiles_per_row) {
    using L = LayoutS<NB, C>;
    constexpr int NW = 8;                          // waves per block, one tile each
    constexpr int NO = L::NO, KC = L::KC, W = 32 * NB;
    constexpr int STRIDE = (W + 63) / 64 * 64;     // floats per vector row: whole 256-B copies
    constexpr int NS = 2 * KC;                     // streamed slabs per pass
    // each wave copies the same number of 1 KB pieces of every slab (repeating
    // a piece where there are fewer than waves), so that a wave's own count
    // of outstanding copies says which slab has landed
    constexpr int PER_WAVE = (L::SLAB / 64 + NW - 1) / NW;
    static_assert(C == 4, "layer 1 is one 16x16x4 fp32 MFMA per output block");
    __shared__ h8 res[L::RES];
    // three buffers: the slab in use and the next two (one array: the copies
    // into it are invisible to the compiler, so nothing is serialised by it)
    __shared__ h8 slabs[3 * L::SLAB];
    __shared__ __attribute__((aligned(16))) float vec[(NW + 2) * STRIDE];   // shifts, b2, b3

    const int groups = src.active ? *src.active : src.max_groups;
    const int64_t ntiles = (int64_t)groups * src.group * tiles_per_row;
    const int64_t ngroups = (ntiles + NW - 1) / NW;
    if ((int64_t)blockIdx.x >= ngroups) return;              // uniform over the block

    const int tid = threadIdx.x, lane = tid & 63, lg = lane >> 4, lj = lane & 15;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t P = a.P;

    // n_units (a multiple of 64) 16-B units of the packed weights -> LDS, 1 KB per wave op
    auto dma = [&](h8* dst, int off, int n_units) {
        const char* gb = reinterpret_cast<const char*>(a.frags);
        uint32_t lo = (uint32_t)lane * 16u;
        asm volatile("" : "+s"(gb), "+v"(lo));
        const uint32_t base = lds_addr(dst);
        for (int c = wave; c < n_units / 64; c += NW)
            dma16(gb + (size_t)(off + c * 64) * 16u, lo, base + (uint32_t)c * 1024u);
    };
    auto slab_buf = [&](int buf) -> h8* { return slabs + buf * L::SLAB; };
    // streamed slab s (0 <= s < NS) -> buffer buf, PER_WAVE copies per wave
    auto dma_slab = [&](int s, int buf) {
        // the empty asm makes the base opaque: the copies' addresses are then
        // formed where they are used, not hoisted out of the loops (where they
        // would hold a hundred registers)
        const char* gb = reinterpret_cast<const char*>(a.frags);
        uint32_t lo = (uint32_t)lane * 16u;
        asm volatile("" : "+s"(gb), "+v"(lo));
        const uint32_t base = lds_addr(slab_buf(buf));
        const int off = L::mid(0, 0) + s * L::SLAB;
#pragma unroll
        for (int i = 0; i < PER_WAVE; ++i) {
            int c = wave + i * NW;
            c = c < L::SLAB / 64 ? c : L::SLAB / 64 - 1;
            dma16(gb + (size_t)(off + c * 64) * 16u, lo, base + (uint32_t)c * 1024u);
        }
    };
    // this wave's first-layer shift (b1 + e_n, plus Wc c on the guided branch) -> its vector row
    // 16 B per lane while a whole 256 floats remain, then 4 B per lane (lanes
    // past the row re-read its last value into the row's padding)
    auto dma_shift = [&](int n, int br) {
        const float* row = (br == 0 ? a.shift_u : a.shift_c) + (int64_t)n * W;
        const uint32_t base = lds_addr(vec + wave * STRIDE);
        constexpr int N4 = W / 256;
        for (int c = 0; c < N4; ++c) dma16(row, (uint32_t)(c * 256 + lane * 4) * 4u, base + (uint32_t)c * 1024u);
        for (int c = N4 * 4; c < STRIDE / 64; ++c) {
            int off = c * 64 + lane;
            off = off < W ? off : W - 1;
            dma4(row, (uint32_t)off * 4u, base + (uint32_t)c * 256u);
        }
    };
    auto land = [&]() {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
    };
    // every copy but this wave's last PER_WAVE (the slab after the one needed) has landed
    auto land_but_next = [&]() {
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"(PER_WAVE) : "memory");
        __syncthreads();
    };
    auto mfma = [](const h8& w, const h8& x, const f4& c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(w, x, c, 0, 0, 0);
    };
    // the weight fragments w0, w1 of output blocks o and o + 1 (at fr, fr + 128),
    // and their three split products
    struct Frag2 {
        h8 a0, a1, b0, b1;
    };
    auto load2 = [](const h8* fr) -> Frag2 { return Frag2{fr[0], fr[64], fr[128], fr[192]}; };
    auto mac3x2 = [&](const Frag2& f, const SplitB& b, f4& A, f4& B) {
        const h8 p0 = __builtin_bit_cast(h8, b.p0), p1 = __builtin_bit_cast(h8, b.p1),
                 p2 = __builtin_bit_cast(h8, b.p2);
        A = mfma(f.a0, p0, A);
        B = mfma(f.b0, p0, B);
        A = mfma(f.a0, p1, A);
        B = mfma(f.b0, p1, B);
        A = mfma(f.a1, p2, A);
        B = mfma(f.b1, p2, B);
    };
    auto mac3 = [&](const h8* fr, const SplitB& b, f4& A) {
        const h8 a0 = fr[0], a1 = fr[64];
        A = mfma(a0, __builtin_bit_cast(h8, b.p0), A);
        A = mfma(a0, __builtin_bit_cast(h8, b.p1), A);
        A = mfma(a1, __builtin_bit_cast(h8, b.p2), A);
    };
    // per-tile scale of a layer's input from its largest |t| (over the wave):
    // S = 2^(11-e) puts S |t| in [2^14, 2^15), so S |u| = S |t| / log2(e) stays
    // below 2^15; a non-finite or zero maximum keeps e = 0 (non-finite values
    // then propagate as in fp32)
    auto scale_of = [&](const f4 (&t)[NO]) -> int {
        float m = 0.f;
        static_for<NO>([&](auto oc) {
            constexpr int o = decltype(oc)::value;
            m = __builtin_fmaxf(m, __builtin_fmaxf(__builtin_fmaxf(__builtin_fabsf(t[o][0]), __builtin_fabsf(t[o][1])),
                                                   __builtin_fmaxf(__builtin_fabsf(t[o][2]), __builtin_fabsf(t[o][3]))));
        });
        m = wave_max_dpp(m);
        int e = 0;
        if (m > 0.f && m <= 3.4028235e38f) {
            const int be = (int)((__builtin_bit_cast(uint32_t, m) >> 23) & 0xff);
            e = (be == 0 ? -126 : be - 127) - 3;
            e = e < -100 ? -100 : (e > 120 ? 120 : e);   // S and 1/S stay normal
        }
        return __builtin_amdgcn_readfirstlane(e);
    };
    struct Tile {
        int64_t row;
        bool active;
        const float* x;
        int n, px;
    };
    auto locate = [&](int64_t tg) -> Tile {
        Tile T;
        const int64_t t = tg * NW + wave;
        T.active = t < ntiles;
        const int64_t tt = T.active ? t : ntiles - 1;       // idle waves redo the last tile
        T.row = tt / tiles_per_row;
        const int pt = (int)(tt % tiles_per_row);
        const int g = (int)(T.row / src.group), bb = (int)(T.row % src.group);
        const int64_t sl = src.slot ? __builtin_amdgcn_readfirstlane(src.slot[g]) : g;
        T.x = src.base + sl * src.slot_stride + (int64_t)bb * C * P;
        T.n = __builtin_amdgcn_readfirstlane(row_timestep(src, g));
        T.px = pt * 16 + lj;
        return T;
    };
    // layer-1 input: lane l carries channel l/16 of pixel l%16
    auto load_x = [&](const Tile& T) -> float { return T.px < P ? T.x[(int64_t)lg * P + T.px] : 0.f; };
    constexpr int nbranch = GUIDED ? 2 : 1;

    Tile cur = locate(blockIdx.x);
    dma(res, 0, L::RES);
    dma_shift(cur.n, 0);
    dma_slab(0, 0);
    dma_slab(1, 1);
    for (int i = tid; i < W; i += NW * 64) {
        vec[NW * STRIDE + i] = a.b2[i];
        vec[(NW + 1) * STRIDE + i] = a.b3[i];
    }
    land();
    float xin = load_x(cur);
    // slab s of the current pass sits in buffer (rot + s) % 3
    int rot = 0;

    for (int64_t tg = blockIdx.x; tg < ngroups; tg += gridDim.x) {
        const bool last_group = tg + gridDim.x >= ngroups;
        const int64_t tg_next = last_group ? tg : tg + gridDim.x;
        f4 eu = f4{0.f, 0.f, 0.f, 0.f};
        float xnx = 0.f;
        for (int br = 0; br < nbranch; ++br) {
            f4 acc[NO], t[NO];
            // ---- layer 1: t = kNegLog2e (W1 x + shift) (fp32 MFMA), from the
            // resident fragments; the shift row holds kNegLog2e (b1 + e_n [+ Wc c])
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // this wave's shift row
            {
                const float* a1 = reinterpret_cast<const float*>(res) + lane;
                const float* sh = vec + wave * STRIDE + 4 * lg;
                static_for<NO>([&](auto oc) {
                    constexpr int o = decltype(oc)::value;
                    const f4 c1 = __builtin_amdgcn_mfma_f32_16x16x4f32(a1[o * 64], xin, f4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
                    const f4 sv = *reinterpret_cast<const f4*>(sh + 16 * o);
#pragma unroll
                    for (int r = 0; r < 4; ++r) t[o][r] = __builtin_fmaf(c1[r], kNegLog2e, sv[r]);
                });
            }
            int e = scale_of(t);
            float invS = pow2(e - 11);
            float cS = kNegLog2e * invS;                  // exact: a power-of-two scaling
            SplitB b = silu_split(t[0], t[1], cS);

            // ---- layers 2 and 3: one streamed slab per reduction chunk
            static_for<2>([&](auto lc) {
                constexpr int layer = decltype(lc)::value;
                static_for<NO>([&](auto oc) { acc[decltype(oc)::value] = f4{0.f, 0.f, 0.f, 0.f}; });
                static_for<KC>([&](auto cc) {
                    constexpr int c = decltype(cc)::value;
                    constexpr int s = layer * KC + c;
                    const int buf = (rot + s) % 3;
                    // slab s has landed (at s = 0 everything has: slabs 0 and 1 were
                    // copied during the previous pass); the buffer of slab s - 1
                    // is free for slab s + 2.  Only the copies of slab s + 1 may
                    // still be in flight; after the last slab of the last pass
                    // none were issued, so nothing may be
                    const bool more = br + 1 < nbranch || !last_group;
                    if constexpr (s == 0) land();
                    else if constexpr (s + 1 == NS) { if (more) land_but_next(); else land(); }
                    else land_but_next();
                    const int nbuf = (rot + s + 2) % 3;
                    if constexpr (s + 2 < NS) {
                        dma_slab(s + 2, nbuf);
                    } else {                                 // the next pass's slabs 0 and 1
                        if (more) {
                            if constexpr (s + 2 == NS) {
                                if (br + 1 < nbranch) dma_shift(cur.n, br + 1);
                                else dma_shift(locate(tg_next).n, 0);
                            }
                            dma_slab(s + 2 - NS, nbuf);
                        }
                    }
                    // software pipeline: the fragments of pair j + 1 are loaded and
                    // one of the nine steps of the next chunk's SiLU and split is
                    // done before the six MFMAs of pair j (the order is fixed: the
                    // scheduler keeps the loads ahead of the products they feed)
                    SplitB bn;
                    SplitR sr;
                    const h8* fr = slab_buf(buf) + lane;
                    Frag2 cur2 = load2(fr);
                    static_for<NO / 2>([&](auto pc) {
                        constexpr int j = decltype(pc)::value;
                        Frag2 nxt2;
                        if constexpr (j + 1 < NO / 2) nxt2 = load2(fr + (2 * j + 2) * 128);
                        if constexpr (c + 1 < KC && j < 9) silu_split_step(j, t[2 * c + 2], t[2 * c + 3], cS, bn, sr);
                        mac3x2(cur2, b, acc[2 * j], acc[2 * j + 1]);
                        // issue order inside the group: each MFMA followed by a
                        // fragment load and one VALU instruction (a vector
                        // instruction beside each matrix one hides behind it; more
                        // than two per MFMA largely serialise with them)
                        static_for<4>([&](auto) {
                            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
                            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // DS read
                            __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);   // VALU
                        });
                        static_for<2>([&](auto) {
                            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                            __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);
                        });
                        __builtin_amdgcn_sched_barrier(0);
                        if constexpr (j + 1 < NO / 2) cur2 = nxt2;
                    });
                    if constexpr (c + 1 < KC) {
                        if constexpr (NO / 2 < 9) {          // fewer pairs than steps
                            static_for<9>([&](auto qc) {
                                if constexpr (decltype(qc)::value >= NO / 2)
                                    silu_split_step(decltype(qc)::value, t[2 * c + 2], t[2 * c + 3], cS, bn, sr);
                            });
                        }
                        b = bn;
                    }
                });
                // epilogue: t = kNegLog2e (acc / S + bias) = acc (kNegLog2e / S) +
                // kNegLog2e bias, the scaling exact, the bias row pre-multiplied
                const float cs = cS;
                const float* bias = vec + (NW + layer) * STRIDE + 4 * lg;
                static_for<NO>([&](auto oc) {
                    constexpr int o = decltype(oc)::value;
                    const f4 bv = *reinterpret_cast<const f4*>(bias + 16 * o);
#pragma unroll
                    for (int r = 0; r < 4; ++r) t[o][r] = __builtin_fmaf(acc[o][r], cs, bv[r]);
                });
                e = scale_of(t);
                invS = pow2(e - 11);
                cS = kNegLog2e * invS;
                b = silu_split(t[0], t[1], cS);
            });

            rot = (rot + NS) % 3;
            if (br + 1 == nbranch) xnx = load_x(locate(tg_next));
            // ---- layer 4 (C outputs in one block, rows past C zero), resident fragments
            f4 o4 = f4{0.f, 0.f, 0.f, 0.f};
            {
                const h8* f4r = res + L::L1 + lane;
                static_for<KC>([&](auto cc) {
                    constexpr int c = decltype(cc)::value;
                    if constexpr (c > 0) b = silu_split(t[2 * c], t[2 * c + 1], cS);
                    mac3(f4r + c * 128, b, o4);
                });
            }
            // lanes 0..15 hold channel r of pixel l in register r
            if (lane < 16) {
                float* out = eps + cur.row * (int64_t)C * P;
#pragma unroll
                for (int r = 0; r < C; ++r) {
                    const float v = __builtin_fmaf(o4[r], invS, a.b4[r]);
                    const bool store = cur.active && cur.px < P;
                    if constexpr (!GUIDED) {
                        if (store) out[(int64_t)r * P + cur.px] = v;
                    } else if (br == 0) {
                        eu[r] = v;
                    } else if (store) {
                        out[(int64_t)r * P + cur.px] = eu[r] + a.guidance * (v - eu[r]);
                    }
                }
            }
        }
        cur = locate(tg_next);
        xin = xnx;
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
void pack_s_t(const float* W1, const float* W2, const float* W3, const float* W4,
              std::vector<uint8_t>& out) {
    using L = LayoutS<NB, C>;
    constexpr int W = 32 * NB;
    out.assign((size_t)L::TOTAL * 16, 0);
    float* f = reinterpret_cast<float*>(out.data());
    for (int o = 0; o < L::NO; ++o)
        for (int l = 0; l < 64; ++l) f[o * 64 + l] = W1[(16 * o + l % 16) * C + l / 16];
    uint16_t* h = reinterpret_cast<uint16_t*>(out.data());
    // element u of lane l in reduction chunk c: input 32 c + 16 (u/4) + 4 (l/16) + u%4
    auto fin = [](int c, int l, int u) { return 32 * c + 16 * (u / 4) + 4 * (l / 16) + u % 4; };
    auto put = [&](int unit, int u, float w) {                  // parts 0, 1 -> units unit, unit + 64
        uint16_t pr[2];
        split_f16(w, pr);
        for (int k = 0; k < 2; ++k) h[((size_t)unit + (size_t)k * 64) * 8 + u] = pr[k];
    };
    for (int c = 0; c < L::KC; ++c)
        for (int l = 0; l < 64; ++l)
            for (int u = 0; u < 8; ++u)
                put(L::L1 + c * 128 + l, u, (l % 16) < C ? W4[(size_t)(l % 16) * W + fin(c, l, u)] : 0.f);
    for (int layer = 0; layer < 2; ++layer) {
        const float* Wm = layer == 0 ? W2 : W3;
        for (int c = 0; c < L::KC; ++c)
            for (int o = 0; o < L::NO; ++o)
                for (int l = 0; l < 64; ++l)
                    for (int u = 0; u < 8; ++u)
                        put(L::mid(layer, c) + o * 128 + l, u, Wm[(size_t)(16 * o + l % 16) * W + fin(c, l, u)]);
    }
}

template <int NB, int C>
void launch_s_t(const ConvArgs& a, const RowSrc& src, float* eps, hipStream_t s) {
    const int tiles_per_row = (int)((a.P + 15) / 16);
    const int64_t ntiles = (int64_t)src.max_groups * src.group * tiles_per_row;
    if (ntiles == 0) return;
    int64_t blocks = (ntiles + 7) / 8;                       // persistent: one block per CU
    if (blocks > device_cus()) blocks = device_cus();
    if (a.shift_c)
        hipLaunchKernelGGL((k_conv_f32s<NB, C, true>), dim3((unsigned)blocks), dim3(512), 0, s, a, src, eps,
                           tiles_per_row);
    else
        hipLaunchKernelGGL((k_conv_f32s<NB, C, false>), dim3((unsigned)blocks), dim3(512), 0, s, a, src, eps,
                           tiles_per_row);
    PD_HIP(hipGetLastError());
}

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
        return bf16 ? (size_t)ConvLayoutBf16<nb, c>::TOTAL * 16 : (size_t)LayoutS<nb, c>::TOTAL * 16;
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
            pack_s_t<nb, c>(W1, W2, W3, W4, out);                 \
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
            launch_s_t<nb, c>(a, src, eps, s);                     \
        return;                                                    \
    }
    PD_CONV_SHAPES(X)
#undef X
    fail(PD_ERR_UNSUPPORTED, "conv1x1: unsupported channel count / width");
}

}  // namespace pd
