// Weight-streaming skinny-M GEMM on MFMA with fused epilogues.
//
// Y[n][m] = sum_k W[n][k] * X[m][k] for the 16*F weight rows of one workgroup
// and the 16*MT tokens of one M block.  At M <= 64 every weight byte is used by
// at most 64 tokens, so the kernel is bound by streaming W from HBM: each wave
// walks a contiguous K range of its F row tiles with D chunks (1 KiB per tile)
// of loads in flight, accumulates on v_mfma 16x16, and the NW waves of the
// workgroup combine their partial sums in LDS in a fixed order (deterministic).
// The finished tile goes to an epilogue functor that applies the op the
// projection feeds (RoPE + KV write, residual, SwiGLU, LM-head reduction).
//
// Row scales (int8 weights) multiply Y per weight row (they factor out of the K
// sum), and row biases (Q/K/V projections) are added after them.  The A operand
// arrives already normalised (RMSNorm applied by the kernel that finished the
// residual row).
#pragma once

#include <type_traits>

#include "common.hpp"

namespace dllm {

struct GemmArgs {
    const void* W;        // packed weights
    const float* wscale;  // per packed row (int8) or nullptr
    const void* X;        // activation fragments
    int KCw;              // weight chunks per row tile
    int KCx;              // activation chunks per token tile
    int n_tiles;          // packed rows / 16
    const float* bias = nullptr;  // per packed row (added after the row scale) or nullptr
    int tpg = 0;          // row tiles per wave group (1 .. FW); the launch sets it
    const uint16_t* qs = nullptr;  // Q4_0: fp16 scales [tile][chunk][16 rows][2 blocks]
    // RMSNorm folded into the GEMM: the operand X holds x * g (not normalised) and the
    // producer left per-group partial sums of x^2, ssq[m * ssq_ld + p] for p < nssq
    // (ssq_ld a multiple of 4); the kernel sums them per token (fixed order) and scales
    // Y[n][m] by rsqrt(sum / dnorm + eps)
    const float* ssq = nullptr;
    int nssq = 0;
    int ssq_ld = 0;
    int dnorm = 0;
    float eps = 0.f;
};

// Epilogue interface:
//   static constexpr int kSmem                      LDS bytes the epilogue keeps per row group
//   struct Pre                                      registers its prologue carries (may be empty)
//   void fetch(Pre& p, int n0, int nrows, int m0, int mcols) const
//       global loads of tables the epilogue needs, issued by every thread before the
//       first weight loads
//   void stage(const Pre& p, char* sm, int n0, int nrows, int m0, int mcols) const
//       stores them to sm once the first weight loads are in flight
//   template <class SC> void operator()(float* Y, int ldy, int n0, int nrows, int m0, int mcols, int part,
//                                       char* sm, const SC& sc) const
// Y is LDS [nrows][ldy] holding the K sums of weight rows [n0, n0 + nrows) for
// tokens [m0, m0 + mcols); the output of row nl, token ml is sc(Y[nl][ml], nl, ml)
// (int8 row scale, folded RMSNorm scale, bias).  Every thread of the workgroup calls
// it (it may use __syncthreads and overwrite Y); `part` numbers the row group for
// per-group partial results.

// No scales at all (most bf16 launches): the epilogues read the sums unchanged.
struct NoScale {
    __device__ __forceinline__ float operator()(float y, int, int) const { return y; }
};

// The scales of a tile's outputs, applied where an epilogue reads Y: a separate pass
// over Y, with its barrier and its per-element loads of the row scales from global
// memory, made the int8 LM head 170 us instead of 159 and the int8 64-row window at
// prefix 4096 4.90 ms instead of 4.74.  The row scales and biases are staged in LDS
// while the weights stream.  Per output: y * ws[nl] (int8 row scale), * rs[ml] (folded
// RMSNorm), + b[nl] (bias); each pointer is to LDS, or nullptr when that scale is
// absent.
struct YScale {
    const float* ws = nullptr;
    const float* rs = nullptr;
    const float* b = nullptr;
    __device__ __forceinline__ float operator()(float y, int nl, int ml) const {
        if (ws != nullptr) y *= ws[nl];
        if (rs != nullptr) y *= rs[ml];
        if (b != nullptr) y += b[nl];
        return y;
    }
};

// Loads in flight per wave: as many K chunks as fit in ~128 VGPRs of buffers.
template <int WT, int F, int MT>
constexpr int pipeline_depth() {
    constexpr int XP = (WT == WT_F32) ? 1 : 2;
    // one row tile per wave (whole-K residual projections): 16 weight stages, the
    // activations at a quarter to a sixteenth of that depth (activation_depth)
    if constexpr (F == 1 && (WT == WT_BF16 || WT == WT_I8)) return 16;
    if constexpr (WT == WT_Q4) {
        // code stages: 8-byte codes + a scale dword per tile (3 VGPRs); the
        // activations have their own, shallower pipeline (activation_depth), so the
        // codes can run deeper: ~64 VGPRs of them up to 2 token tiles (an even count),
        // ~36 at 3 and one stage at 4 token tiles
        if constexpr (MT <= 2) {
            constexpr int d = 64 / (3 * F);
            return d < 2 ? 2 : (d > 8 ? 8 : (d & ~1));
        } else {
            constexpr int d = (MT == 3 ? 36 : 12) / (3 * F);
            return d < 1 ? 1 : (d > 8 ? 8 : d);
        }
    }
    // bf16 at 3-4 token tiles (row groups of 2-6 tiles): the activation stages take
    // most of the registers (2 planes x MT tiles), so one activation stage (L2-resident)
    // beside 3-4 weight stages (HBM) instead of 2-3 of each (activation_depth);
    // LLaDA-8B, 64-row window at prefix 1024: 5.25 -> 5.16 ms per step
    if constexpr (WT == WT_BF16 && MT >= 3 && F > 1 && F < 8) return (MT == 4 || F == 6) ? 3 : 4;
    constexpr int slot = 4 * (F + MT * WTraits<WT>::XPER * XP);
    constexpr int d = 128 / slot;
    return d < 1 ? 1 : (d > 8 ? 8 : d);
}

// Activation stages in flight: the weight depth, except for Q4_0 whose code
// pipeline runs deeper than its activations (L2-resident, 16 dwords per token tile
// and stage): one stage, which leaves the registers for 6 row tiles per wave
// (LLaDA-8B gate/up at 32 rows: 23.6 us per launch against 33.5 with 3 tiles and
// two activation stages); and bf16 at 3-4 token tiles (pipeline_depth).
template <int WT, int F, int MT>
constexpr int activation_depth() {
    if constexpr (WT == WT_Q4) return 1;
    if constexpr (WT == WT_BF16 && MT >= 3 && F > 1 && F < 8) return (MT == 4 || F == 6) ? 1 : 2;
    // the 10-tile gate/up (Dream-7B widths): one activation stage beside two weight
    // stages; with two of each it spilled (gate/up 53.4 -> 51.4 us, step 3.95 -> 3.85 ms)
    if constexpr (WT == WT_BF16 && F == 10 && MT <= 2) return 1;
    if constexpr (F == 1 && (WT == WT_BF16 || WT == WT_I8)) {
        // ~64 VGPRs of activation stages (hi + lo planes, XPER 32-column halves)
        constexpr int per = 4 * WTraits<WT>::XPER * 2 * MT;
        constexpr int d = 64 / per;
        return d >= 8 ? 8 : (d >= 4 ? 4 : (d >= 2 ? 2 : 1));
    }
    return pipeline_depth<WT, F, MT>();
}


// Reduction slots: the largest power of two <= NWk whose slots fit ~150 KiB of LDS (a
// workgroup of these layouts has its CU to itself).  With one slot per wave the
// K-slice sums take one write round: LLaDA-8B down at 32 rows (8 slots of 16.5 KiB)
// 26.9 -> 26.2 us, 32-row step at prefix 512 3.99 -> 3.97 ms, against a 100 KiB budget.
template <int NWk>
constexpr int reduce_slots(int slot_bytes) {
    int s = NWk;
    while (s > 1 && s * slot_bytes > 150 * 1024) s >>= 1;
    return s;
}

// Workgroup layout: NWn x NWk waves.  Wave (wn, wk) streams g.tpg <= FW row tiles
// (group wn) over slice wk of the workgroup's K range; the NWk slices of a group are
// summed in LDS in a fixed order.  grid = (row groups / NWn, KS, token blocks):
// blockIdx.y picks one of KS contiguous K ranges (split-K; the partial results
// go to an epilogue that stores them for a separate reduction).
template <int WT, int FW, int NWn, int NWk, int MT, class Epi>
__global__ void __launch_bounds__(NWn * NWk * 64)
gemm_kernel(GemmArgs g, Epi epi) {
    constexpr int XPER = WTraits<WT>::XPER;
    constexpr bool XF = (WT == WT_F32);
    constexpr int XP = XF ? 1 : 2;                 // activation planes (hi, lo)
    constexpr int XB = XChunk<XF>::bytes;
    constexpr int D = pipeline_depth<WT, FW, MT>();
    constexpr int DX = activation_depth<WT, FW, MT>();
    static_assert(D % DX == 0, "activation stages must divide the weight stages");
    constexpr int NW = NWn * NWk;
    constexpr int NR = 16 * FW, MR = 16 * MT, LDY = MR + 1;
    // K-slice partials: S slots per row group (S <= NWk, a power of two that keeps
    // the workgroup's slots within ~150 KiB of LDS); slot 0 ends with the sum.
    constexpr int SLOT = NR * LDY;
    constexpr int S = reduce_slots<NWk>(NWn * SLOT * 4);
    __shared__ float Y[NWn][S * SLOT];
    constexpr int ESM = Epi::kSmem > 0 ? Epi::kSmem : 16;
    __shared__ __align__(16) char esm[NWn * ESM];
    __shared__ float rs_sm[MR];                    // folded RMSNorm: rsqrt(mean x^2 + eps) per token
    __shared__ float ws_sm[NWn][NR];               // int8 row scales of each group's rows
    __shared__ float b_sm[NWn][NR];                // biases of each group's rows

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int wn = wave % NWn, wk = wave / NWn;
    // Token blocks (grid.z > 1: windows of 65-512 rows).  The dispatcher deals
    // consecutive workgroups to the 8 XCDs in turn; this mapping gives the z blocks
    // of one row group consecutive slots on one XCD, so they run together and the
    // group's weights come from HBM once and from that XCD's L2 after (LLaDA-8B
    // gate/up at 512 rows: 270 against 358 us).  Past 8 blocks their activations
    // no longer fit beside the weights and plain order is faster.
    int bx = blockIdx.x, bz = blockIdx.z;
    if (gridDim.z > 1 && gridDim.z <= 8 && gridDim.y == 1 && (gridDim.x & 7) == 0) {
        const unsigned L = blockIdx.x + gridDim.x * blockIdx.z, j = L >> 3;
        bx = (int)((j / gridDim.z) * 8 + (L & 7));
        bz = (int)(j % gridDim.z);
    }
    const int mt0 = bz * MT;
    // K range of this split (32-bit unsigned: KCw * KS is far below 2^32, and a 64-bit
    // division would delay the first weight load by a few hundred scalar instructions)
    const unsigned KS = gridDim.y, KCw = (unsigned)g.KCw;
    const int kb0 = KS == 1 ? 0 : (int)((blockIdx.y * KCw) / KS);
    const int kb1 = KS == 1 ? g.KCw : (int)(((blockIdx.y + 1) * KCw) / KS);

    typename Epi::Pre pre[NWn];
#pragma unroll
    for (int q = 0; q < NWn; ++q) {
        const int nq0 = (bx * NWn + q) * g.tpg;
        const int nfq = max(0, min(g.tpg, g.n_tiles - nq0));
        if (nfq > 0) epi.fetch(pre[q], nq0 * 16, nfq * 16, mt0 * 16, MR);
    }
    // row scales and biases of the groups' rows: loaded before the weights, stored to
    // LDS with the epilogue's tables
    constexpr int NSC = (NWn * NR + NWn * NWk * 64 - 1) / (NWn * NWk * 64);
    const bool has_rowsc = g.wscale != nullptr || g.bias != nullptr;
    float scv[NSC], biv[NSC];
    if (has_rowsc) {
#pragma unroll
        for (int j = 0; j < NSC; ++j) {
            const int idx = threadIdx.x + j * NWn * NWk * 64;
            const int q = idx / NR, nl = idx % NR;
            const int row = (bx * NWn + q) * g.tpg * 16 + nl;
            const bool ok = idx < NWn * NR && nl < 16 * g.tpg && row < 16 * g.n_tiles;
            scv[j] = (ok && g.wscale != nullptr) ? g.wscale[row] : 1.f;
            biv[j] = (ok && g.bias != nullptr) ? g.bias[row] : 0.f;
        }
    }
    auto stage_prologue = [&]() {
#pragma unroll
        for (int q = 0; q < NWn; ++q) {
            const int nq0 = (bx * NWn + q) * g.tpg;
            const int nfq = max(0, min(g.tpg, g.n_tiles - nq0));
            if (nfq > 0) epi.stage(pre[q], esm + q * ESM, nq0 * 16, nfq * 16, mt0 * 16, MR);
        }
        if (has_rowsc) {
#pragma unroll
            for (int j = 0; j < NSC; ++j) {
                const int idx = threadIdx.x + j * NWn * NWk * 64;
                if (idx < NWn * NR) {
                    ws_sm[idx / NR][idx % NR] = scv[j];
                    b_sm[idx / NR][idx % NR] = biv[j];
                }
            }
        }
    };

    f32x4_t acc[FW][MT];
#pragma unroll
    for (int f = 0; f < FW; ++f)
#pragma unroll
        for (int t = 0; t < MT; ++t) acc[f][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    {
        const int nt0 = (bx * NWn + wn) * g.tpg;
        const int nf = max(0, min(g.tpg, g.n_tiles - nt0));
        const unsigned span = (unsigned)(kb1 - kb0);
        const int c0 = kb0 + (int)(((unsigned)wk * span) / NWk);
        const int c1 = kb0 + (int)(((unsigned)(wk + 1) * span) / NWk);
        constexpr int WCB = wchunk_bytes<WT>();
        const char* wp = (const char*)g.W + ((size_t)nt0 * g.KCw * 64 + lane) * (WCB / 64);
        const char* xp = (const char*)g.X + (size_t)mt0 * g.KCx * XB + lane * 16;
        const size_t wtile = (size_t)g.KCw * WCB, xtile = (size_t)g.KCx * XB;
        // Q4_0 scales of this lane's row: one dword (two fp16) per chunk
        [[maybe_unused]] const uint32_t* qsp =
            (WT == WT_Q4) ? (const uint32_t*)g.qs + (size_t)nt0 * g.KCw * 16 + (lane & 15) : nullptr;

        u32x4_t wb[D][FW];                    // weight chunks (bf16 / int8 / fp32)
        [[maybe_unused]] u32x2_t wq[D][FW];   // Q4_0 codes
        [[maybe_unused]] uint32_t wsc[D][FW]; // Q4_0 scales (two fp16)
        u32x4_t xb[DX][MT * XPER * XP];

        // full (std::true_type): the group fills the template, no tile needs a condition
        auto loadw_t = [&](int s, int c, auto full) {
#pragma unroll
            for (int f = 0; f < FW; ++f) {
                if constexpr (!decltype(full)::value) {
                    if (f >= nf) continue;
                }
                if constexpr (WT == WT_Q4) {
                    wq[s][f] = ldg8_nt(wp + f * wtile + (size_t)c * WCB);
                    wsc[s][f] = qsp[((size_t)f * g.KCw + c) * 16];
                } else {
                    wb[s][f] = ldg16_nt(wp + f * wtile + (size_t)c * WCB);
                }
            }
        };
        auto loadw = [&](int s, int c) { loadw_t(s, c, std::false_type{}); };
        auto loadx = [&](int s, int c) {
#pragma unroll
            for (int t = 0; t < MT; ++t)
#pragma unroll
                for (int h = 0; h < XPER; ++h)
#pragma unroll
                    for (int pl = 0; pl < XP; ++pl)
                        xb[s][(t * XPER + h) * XP + pl] =
                            ldg16(xp + t * xtile + (size_t)(c * XPER + h) * XB + pl * 1024);
        };
        auto compute = [&](int s, int sx) {
            // Q4_0 (weights as the B operand, so a lane's accumulator column is one
            // weight row and takes one scale per block): codes unpack to bf16 128 + q,
            // so a block's MFMAs start from zp = -136 * sum_k x and give
            // sum_k (q - 8) x exactly up to fp32 accumulation; then acc += d * that.
            if constexpr (WT == WT_Q4) {
                const u32x4_t ones = {0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u};   // bf16 1.0
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    f32x4_t zp[MT];
#pragma unroll
                    for (int t = 0; t < MT; ++t) {
                        f32x4_t z = mfma_bf16(xb[sx][(t * 2 + h) * 2 + 0], ones, f32x4_t{0.f, 0.f, 0.f, 0.f});
                        z = mfma_bf16(xb[sx][(t * 2 + h) * 2 + 1], ones, z);
#pragma unroll
                        for (int i = 0; i < 4; ++i) zp[t][i] = -136.0f * z[i];
                    }
#pragma unroll
                    for (int f = 0; f < FW; ++f) {
                        // at 3-4 token tiles the Q4_0 chains of all tiles do not fit the
                        // registers together: one tile at a time
                        if constexpr (MT >= 3) {
                            if (f >= nf) continue;
                        }
                        const float sc = f16_bits_to_f32(h == 0 ? (wsc[s][f] & 0xFFFFu) : (wsc[s][f] >> 16));
                        const u32x4_t w = q4_unpack(wq[s][f][h]);
#pragma unroll
                        for (int t = 0; t < MT; ++t) {
                            f32x4_t v = mfma_bf16(xb[sx][(t * 2 + h) * 2 + 0], w, zp[t]);
                            v = mfma_bf16(xb[sx][(t * 2 + h) * 2 + 1], w, v);
#pragma unroll
                            for (int i = 0; i < 4; ++i) acc[f][t][i] = fmaf(sc, v[i], acc[f][t][i]);
                        }
                    }
                }
                return;
            }
#pragma unroll
            for (int f = 0; f < FW; ++f) {
                if constexpr (WT == WT_BF16) {
#pragma unroll
                    for (int t = 0; t < MT; ++t) {
                        acc[f][t] = mfma_bf16(wb[s][f], xb[sx][t * 2 + 0], acc[f][t]);
                        acc[f][t] = mfma_bf16(wb[s][f], xb[sx][t * 2 + 1], acc[f][t]);
                    }
                } else if constexpr (WT == WT_I8) {
                    const u32x4_t w0 = i8x8_to_bf16x8(wb[s][f][0], wb[s][f][1]);
                    const u32x4_t w1 = i8x8_to_bf16x8(wb[s][f][2], wb[s][f][3]);
#pragma unroll
                    for (int t = 0; t < MT; ++t) {
                        acc[f][t] = mfma_bf16(w0, xb[sx][(t * 2 + 0) * 2 + 0], acc[f][t]);
                        acc[f][t] = mfma_bf16(w0, xb[sx][(t * 2 + 0) * 2 + 1], acc[f][t]);
                        acc[f][t] = mfma_bf16(w1, xb[sx][(t * 2 + 1) * 2 + 0], acc[f][t]);
                        acc[f][t] = mfma_bf16(w1, xb[sx][(t * 2 + 1) * 2 + 1], acc[f][t]);
                    }
                } else {
#pragma unroll
                    for (int t = 0; t < MT; ++t)
#pragma unroll
                        for (int q = 0; q < 4; ++q)
                            acc[f][t] = mfma_f32(__uint_as_float(wb[s][f][q]), __uint_as_float(xb[sx][t][q]),
                                                 acc[f][t]);
                }
            }
        };

        // Every tile slot of the template is computed, without a per-tile branch (a
        // branch per tile splits the unrolled step into basic blocks the scheduler
        // cannot interleave); slots past nf hold zeros (never loaded) and their
        // results are never stored.
#pragma unroll
        for (int s = 0; s < D; ++s)
#pragma unroll
            for (int f = 0; f < FW; ++f) {
                if constexpr (WT == WT_Q4) {
                    wq[s][f] = u32x2_t{0u, 0u};
                    wsc[s][f] = 0u;
                } else {
                    wb[s][f] = u32x4_t{0u, 0u, 0u, 0u};
                }
            }
        // Folded RMSNorm: each wave sums the partials of tokens wave, wave + NW, ... (one
        // token per wave at a time): lane l adds partials 4l .. 4l+3 (+ 256 per further
        // chunk) in order, then a fixed xor tree over the wave, so every workgroup gets
        // the same bits.  The first four tokens' loads go out before the weight loads
        // (the waits count loads in issue order, so consuming them later does not wait
        // for the weight stages).
        float4 ssq_t[4];
        auto ssq_load = [&](int j0) {
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                const int j = j0 + b * NW, p = 4 * lane;
                ssq_t[b] = make_float4(0.f, 0.f, 0.f, 0.f);
                if (j < MR) {
                    const float* row = g.ssq + (size_t)(mt0 * 16 + j) * g.ssq_ld;
                    if (p + 3 < g.nssq) {
                        ssq_t[b] = *(const float4*)(row + p);
                    } else {
                        if (p < g.nssq) ssq_t[b].x = row[p];
                        if (p + 1 < g.nssq) ssq_t[b].y = row[p + 1];
                        if (p + 2 < g.nssq) ssq_t[b].z = row[p + 2];
                    }
                }
            }
        };
        auto ssq_reduce = [&](int j0) {
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                const int j = j0 + b * NW;
                float v = (ssq_t[b].x + ssq_t[b].y) + (ssq_t[b].z + ssq_t[b].w);
                for (int c = 256; c < g.nssq; c += 256) {      // d > 4096: further chunks
                    const float* row = g.ssq + (size_t)(mt0 * 16 + min(j, MR - 1)) * g.ssq_ld + c;
                    for (int e = 0; e < 4; ++e)
                        if (j < MR && c + 4 * lane + e < g.nssq) v += row[4 * lane + e];
                }
                v = warp_sum(v);
                if (j < MR && lane == 0) rs_sm[j] = 1.0f / sqrtf(v / (float)g.dnorm + g.eps);
            }
        };
        if (g.ssq != nullptr) ssq_load(wave);
        const bool work = c1 > c0 && nf > 0;
        if (work) {
#pragma unroll
            for (int s = 0; s < D; ++s) {
                loadw(s, min(c0 + s, c1 - 1));
                if (s < DX) loadx(s, min(c0 + s, c1 - 1));
            }
        }
        stage_prologue();
        if (g.ssq != nullptr) {
            ssq_reduce(wave);
            for (int j0 = wave + 4 * NW; j0 < MR; j0 += 4 * NW) {
                ssq_load(j0);
                ssq_reduce(j0);
            }
        }
        if (work) {
            // chunk c uses weight slot c % D and activation slot c % DX (DX divides D).
            // For a group that fills the template, rounds whose D successors all lie
            // in the K range run without conditions: there the compiler knows how many
            // loads are in flight and each step waits only for its own chunk (with loads
            // behind branches it waits for all but 1-3 of them: one stage of pipeline).
            // LLaDA-8B at 32 rows: gate/up 39.5 -> 37.4 us, down 23.5 -> 22.4 us; int8
            // at 64 rows: gate/up 36.4 -> 34.7 us.  bf16 at 3-4 token tiles and Q4_0
            // were slower with it (64-row bf16 gate/up 46.7 -> 59.8 us, Q4_0 LM head 138
            // -> 193 us), so they keep the conditional steps throughout.
            int base = c0;
            if constexpr (WT == WT_I8 || (WT == WT_BF16 && MT <= 2)) {
                if (nf == FW) {
                    for (; base + 2 * D <= c1; base += D) {
#pragma unroll
                        for (int s = 0; s < D; ++s) {
                            const int c = base + s, sx = s % DX;
                            compute(s, sx);
                            loadw_t(s, c + D, std::true_type{});
                            loadx(sx, c + DX);
                        }
                    }
                    // a last round whose chunks are all loaded: computes only (QKV, O
                    // and down at the LLaDA-8B widths end this way; gate/up's 16 chunks
                    // per wave over 3 stages leave 4, which take the conditional steps)
                    if (c1 - base <= D) {
#pragma unroll
                        for (int s = 0; s < D; ++s) {
                            if (base + s < c1) compute(s, s % DX);
                            // shallower activation stages keep streaming (slot s % DX is free)
                            if constexpr (DX < D) {
                                if (base + s + DX < c1) loadx(s % DX, base + s + DX);
                            }
                        }
                        base = c1;
                    }
                }
            }
            for (; base < c1; base += D) {
#pragma unroll
                for (int s = 0; s < D; ++s) {
                    const int c = base + s, sx = s % DX;
                    if (c < c1) compute(s, sx);
                    if (c + D < c1) loadw(s, c + D);
                    if (c + DX < c1) loadx(sx, c + DX);
                }
            }
        }
    }

    // Sum the NWk K-slices of each row group into Y[wn] in a fixed order: wave wk
    // adds into slot wk % S (rounds of S waves), then every thread sums the S
    // slots of its elements in slot order.
    const int r = lane & 15, gq = lane >> 4;
    for (int k0 = 0; k0 < NWk; k0 += S) {
        if (wk >= k0 && wk < k0 + S) {
            float* slot = &Y[wn][(wk - k0) * SLOT];
#pragma unroll
            for (int f = 0; f < FW; ++f)
#pragma unroll
                for (int t = 0; t < MT; ++t)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        // Q4_0 accumulators are transposed: element i is token 4gq + i of row r
                        float* p = (WT == WT_Q4) ? slot + (16 * f + r) * LDY + 16 * t + 4 * gq + i
                                                 : slot + (16 * f + 4 * gq + i) * LDY + 16 * t + r;
                        *p = (k0 == 0) ? acc[f][t][i] : *p + acc[f][t][i];
                    }
        }
        __syncthreads();
    }
    if constexpr (S > 1) {
        for (int idx = threadIdx.x; idx < NWn * NR * MR; idx += blockDim.x) {
            const int q = idx / (NR * MR), e = idx % (NR * MR);
            const int o = (e / MR) * LDY + e % MR;
            float v = Y[q][o];
#pragma unroll
            for (int sl = 1; sl < S; ++sl) v += Y[q][sl * SLOT + o];
            Y[q][o] = v;
        }
        __syncthreads();
    }

    // The epilogue of each row group, which applies the row scales (int8), the folded
    // RMSNorm scale and the biases as it reads the sums.
    for (int q = 0; q < NWn; ++q) {
        const int nt0 = (bx * NWn + q) * g.tpg;
        const int nf = max(0, min(g.tpg, g.n_tiles - nt0));
        if (nf == 0) break;
        if (has_rowsc || g.ssq != nullptr) {
            YScale sc;
            if (g.wscale != nullptr) sc.ws = ws_sm[q];
            if (g.ssq != nullptr) sc.rs = rs_sm;
            if (g.bias != nullptr) sc.b = b_sm[q];
            epi(Y[q], LDY, nt0 * 16, nf * 16, mt0 * 16, MR, bx * NWn + q, esm + q * ESM, sc);
        } else {
            epi(Y[q], LDY, nt0 * 16, nf * 16, mt0 * 16, MR, bx * NWn + q, esm + q * ESM, NoScale{});
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// Epilogues
// ---------------------------------------------------------------------------

// Q/K/V projection: RoPE on Q and K, Q to a row-major buffer, K and V to the
// cache at each token's position.  Packed rows: [Q | K | V], each d rows; inside
// a Q or K head, packed row 2i is dim i and row 2i+1 is dim i + Dh/2, so a RoPE
// pair is two adjacent rows.  fp32 models store fp32; bf16 / int8 / Q4_0 models
// store K and V as one fp16 plane and Q as an fp16 hi and lo plane (`q_plane`
// elements apart), the operands of the attention's fp16 MFMAs.
template <bool XF32>
struct EpiQKV {
    using T = typename std::conditional<XF32, float, uint16_t>::type;
    int d, dkv, Dh, M;      // Q rows (H * Dh), K and V rows each (Hkv * Dh), head size, real tokens
    int pos_base;           // position of token m is pos ? pos[m] : pos_base + m
    const int* pos;
    const float2* rope;     // [max_pos][Dh/2] (cos, sin)
    T* q;                   // [rows][d] (+ lo plane at q + q_plane)
    size_t q_plane;
    T* Kc;                  // layer base of K   [Hkv][Cs][Dh]
    T* Vt;                  // layer base of V^T [Hkv][Dh][Cs]
    int Cs;

    static constexpr int kPairs = 24 * 64;          // staged (cos, sin): 3 row tiles x 64 tokens
    static constexpr int kSmem = kPairs * 8;

    // one Q value (fp16 hi and lo planes) / one cache value (one fp16 plane)
    __device__ __forceinline__ static void put_q(T* p, size_t plane, float v) {
        if constexpr (XF32) {
            *p = v;
        } else {
            uint16_t hi, lo;
            split_f16(v, hi, lo);
            p[0] = hi;
            p[plane] = lo;
        }
    }
    __device__ __forceinline__ static void put_kv(T* p, float v) {
        if constexpr (XF32) *p = v;
        else *p = f16_sat(v);
    }

    // (cos, sin) of every (pair, token) of the group's Q/K rows: the first kPre per
    // thread go through registers (loaded before the weights), the rest (only for
    // workgroups of fewer than kPairs / kPre threads) are copied directly in stage()
    static constexpr int kPre = 3;
    struct Pre {
        float2 cs[kPre];
    };
    __device__ __forceinline__ bool rope_entry(int idx, int n0, int npairs, int m0, float2& v) const {
        const int p = idx % npairs, ml = idx / npairs;
        const int m = m0 + ml, n = n0 + 2 * p;
        if (m >= M || n >= d + dkv) return false;
        const int rr = n % Dh;                       // d is a multiple of Dh
        const int ps = pos ? pos[m] : pos_base + m;
        v = rope[(size_t)ps * (Dh >> 1) + (rr >> 1)];
        return true;
    }
    __device__ void fetch(Pre& pr, int n0, int nrows, int m0, int mcols) const {
        const int npairs = nrows >> 1, n = npairs * mcols;
        if (n > kPairs) return;
#pragma unroll
        for (int u = 0; u < kPre; ++u) {
            const int idx = threadIdx.x + u * blockDim.x;
            pr.cs[u] = make_float2(0.f, 0.f);
            if (idx < n) rope_entry(idx, n0, npairs, m0, pr.cs[u]);
        }
    }
    __device__ void stage(const Pre& pr, char* sm, int n0, int nrows, int m0, int mcols) const {
        const int npairs = nrows >> 1, n = npairs * mcols;
        if (n > kPairs) return;
        float2* cs = (float2*)sm;
#pragma unroll
        for (int u = 0; u < kPre; ++u) {
            const int idx = threadIdx.x + u * blockDim.x;
            if (idx < n) cs[idx] = pr.cs[u];
        }
        for (int idx = threadIdx.x + kPre * blockDim.x; idx < n; idx += blockDim.x) {
            float2 v;
            if (rope_entry(idx, n0, npairs, m0, v)) cs[idx] = v;
        }
    }

    // four consecutive Q values (fp32: one 16-byte store; else 8-byte hi and lo stores)
    __device__ __forceinline__ static void put4_q(T* p, size_t plane, const float (&v)[4]) {
        if constexpr (XF32) {
            *(float4*)p = make_float4(v[0], v[1], v[2], v[3]);
        } else {
            uint16_t h[4], l[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) split_f16(v[e], h[e], l[e]);
            *(uint2*)p = make_uint2(h[0] | ((uint32_t)h[1] << 16), h[2] | ((uint32_t)h[3] << 16));
            *(uint2*)(p + plane) = make_uint2(l[0] | ((uint32_t)l[1] << 16), l[2] | ((uint32_t)l[3] << 16));
        }
    }
    // four consecutive cache values (fp32: 16 bytes; else one 8-byte fp16 store)
    __device__ __forceinline__ static void put4_kv(T* p, const float (&v)[4]) {
        if constexpr (XF32) {
            *(float4*)p = make_float4(v[0], v[1], v[2], v[3]);
        } else {
            *(uint2*)p = make_uint2(f16_sat(v[0]) | ((uint32_t)f16_sat(v[1]) << 16),
                                    f16_sat(v[2]) | ((uint32_t)f16_sat(v[3]) << 16));
        }
    }

    template <class SC>
    __device__ void operator()(float* Y, int ldy, int n0, int nrows, int m0, int mcols, int, char* sm,
                               const SC& sc) const {
        const int npairs = nrows >> 1;
        const int half = Dh >> 1;
        const bool staged = npairs * mcols <= kPairs;
        const float2* csm = (const float2*)sm;
        if (n0 + nrows <= d + dkv) {
            // Q / K rows: four consecutive RoPE pairs (dims j..j+3 and j+half..j+half+3) per thread
            const int nq = npairs >> 2;
            for (int idx = threadIdx.x; idx < nq * mcols; idx += blockDim.x) {
                const int qd = idx % nq, ml = idx / nq;
                const int m = m0 + ml;
                if (m >= M) continue;
                const int p0 = 4 * qd, n = n0 + 2 * p0;
                const int ps = pos ? pos[m] : pos_base + m;
                const int seg = n < d ? 0 : 1, nn = n - seg * d;
                const int h = nn / Dh, j0 = (nn - h * Dh) >> 1;
                float ra[4], rb[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int na = 2 * (p0 + e);
                    const float a = sc(Y[na * ldy + ml], na, ml), b = sc(Y[(na + 1) * ldy + ml], na + 1, ml);
                    const float2 cs = staged ? csm[p0 + e + npairs * ml] : rope[(size_t)ps * half + j0 + e];
                    ra[e] = a * cs.x - b * cs.y;
                    rb[e] = a * cs.y + b * cs.x;
                }
                if (seg == 0) {
                    T* dst = q + (size_t)m * d + h * Dh;
                    put4_q(dst + j0, q_plane, ra);
                    put4_q(dst + j0 + half, q_plane, rb);
                } else {
                    T* dst = Kc + ((size_t)h * Cs + ps) * Dh;
                    put4_kv(dst + j0, ra);
                    put4_kv(dst + j0 + half, rb);
                }
            }
            return;
        }
        if (n0 >= d + dkv && pos == nullptr && ((pos_base + m0) & 3) == 0) {
            // V^T rows, consecutive positions: four tokens per thread along the row; a
            // quad that reaches past the last real row falls back to single stores
            const int nt = mcols >> 2;
            for (int idx = threadIdx.x; idx < nrows * nt; idx += blockDim.x) {
                const int tq = idx % nt, nl = idx / nt;
                const int m = m0 + 4 * tq;
                if (m >= M) continue;
                const int nn = n0 + nl - d - dkv;
                const int h = nn / Dh, rr = nn - h * Dh;
                T* dst = Vt + ((size_t)h * Dh + rr) * Cs + pos_base + m;
                const float* y = Y + nl * ldy + 4 * tq;
                if (m + 3 < M) {
                    const float v[4] = {sc(y[0], nl, 4 * tq), sc(y[1], nl, 4 * tq + 1), sc(y[2], nl, 4 * tq + 2),
                                        sc(y[3], nl, 4 * tq + 3)};
                    put4_kv(dst, v);
                } else {
                    for (int e = 0; e < 4 && m + e < M; ++e) put_kv(dst + e, sc(y[e], nl, 4 * tq + e));
                }
            }
            return;
        }
        // general case (a group across the K/V boundary, or explicit positions)
        for (int idx = threadIdx.x; idx < npairs * mcols; idx += blockDim.x) {
            const int p = idx % npairs, ml = idx / npairs;
            const int m = m0 + ml;
            if (m >= M) continue;
            const int n = n0 + 2 * p;
            const float a = sc(Y[(2 * p) * ldy + ml], 2 * p, ml), b = sc(Y[(2 * p + 1) * ldy + ml], 2 * p + 1, ml);
            const int ps = pos ? pos[m] : pos_base + m;
            const int seg = n < d ? 0 : (n < d + dkv ? 1 : 2);
            const int nn = n - (seg == 0 ? 0 : (seg == 1 ? d : d + dkv));
            const int h = nn / Dh, rr = nn - h * Dh;
            if (seg < 2) {
                const int j = rr >> 1;
                const float2 cs = staged ? csm[p + npairs * ml] : rope[(size_t)ps * half + j];
                const float ra = a * cs.x - b * cs.y;
                const float rb = a * cs.y + b * cs.x;
                if (seg == 0) {
                    T* dst = q + (size_t)m * d + h * Dh;
                    put_q(dst + j, q_plane, ra);
                    put_q(dst + j + half, q_plane, rb);
                } else {
                    T* dst = Kc + ((size_t)h * Cs + ps) * Dh;
                    put_kv(dst + j, ra);
                    put_kv(dst + j + half, rb);
                }
            } else {
                T* dst = Vt + ((size_t)h * Dh + rr) * Cs + ps;
                put_kv(dst, a);
                put_kv(dst + Cs, b);
            }
        }
    }
};

// Split-K partial results: P[ks][m][n] = Y[n][m] (a reduction kernel finishes them).
struct EpiPartial {
    float* P;
    int ldn;                // row length of P (>= packed rows, a multiple of 4)
    int rows;               // token rows per K slice of P

    static constexpr int kSmem = 0;
    struct Pre {};
    __device__ void fetch(Pre&, int, int, int, int) const {}
    __device__ void stage(const Pre&, char*, int, int, int, int) const {}

    template <class SC>
    __device__ void operator()(float* Y, int ldy, int n0, int nrows, int m0, int mcols, int, char*,
                               const SC& sc) const {
        float* base = P + (size_t)blockIdx.y * rows * ldn;
        const int nq = nrows >> 2;
        for (int idx = threadIdx.x; idx < nq * mcols; idx += blockDim.x) {
            const int qd = idx % nq, ml = idx / nq, nl = 4 * qd;
            const float* y = Y + nl * ldy + ml;
            *(float4*)(base + (size_t)(m0 + ml) * ldn + n0 + nl) =
                make_float4(sc(y[0], nl, ml), sc(y[ldy], nl + 1, ml), sc(y[2 * ldy], nl + 2, ml),
                            sc(y[3 * ldy], nl + 3, ml));
        }
    }
};

// Residual projection over the whole K range (O or down, one 16-row tile per group):
// x[m][n] += Y[n][m] for the group's columns n of the real tokens, then the next
// GEMM's operand u = x * g_next into its fragments and the group's partial sum of
// x^2 per token, ssq[m][grp] (the consumer folds the partials into its RMSNorm
// scale).  Padding tokens get u = 0 and a zero partial.  With `slot` (the last layer
// before a selective LM head) token m's operand and partial go to row slot[m], and
// tokens without a slot write neither.  Each thread takes four
// consecutive columns of one token; the four threads of a token sum their squares by
// a fixed shuffle tree.
template <bool XF32>
struct EpiResidual {
    float* x;               // residual [rows][d]
    int d, M;
    const float* g;         // gain of the next RMSNorm [d]
    void* xg;               // next GEMM's operand fragments (K = d)
    int KCx;
    float* ssq;             // [rows][ssq_ld]: partial of row tile grp at [m * ssq_ld + grp]
    int ssq_ld;
    const int* slot = nullptr;   // operand / partial row of token m (LM-head slots), or identity

    static constexpr int kSmem = 0;
    struct Pre {};
    __device__ void fetch(Pre&, int, int, int, int) const {}
    __device__ void stage(const Pre&, char*, int, int, int, int) const {}

    template <class SC>
    __device__ void operator()(float* Y, int ldy, int n0, int nrows, int m0, int mcols, int grp, char*,
                               const SC& sc) const {
        // nrows is 16 (one row tile): 4 quads per token, consecutive threads
        for (int idx = threadIdx.x; idx < 4 * mcols; idx += blockDim.x) {
            const int qd = idx & 3, ml = idx >> 2;
            const int m = m0 + ml, n = n0 + 4 * qd;
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f), u = v;
            if (m < M && n < d) {
                float4* xp = (float4*)(x + (size_t)m * d + n);
                v = *xp;
                const float* y = Y + (4 * qd) * ldy + ml;
                v.x += sc(y[0], 4 * qd, ml); v.y += sc(y[ldy], 4 * qd + 1, ml);
                v.z += sc(y[2 * ldy], 4 * qd + 2, ml); v.w += sc(y[3 * ldy], 4 * qd + 3, ml);
                *xp = v;
                const float4 gg = *(const float4*)(g + n);
                u = make_float4(v.x * gg.x, v.y * gg.y, v.z * gg.z, v.w * gg.w);
            }
            const int dst = slot != nullptr ? (m < M ? slot[m] : -1) : m;
            if (n < d && dst >= 0) xfrag_store4<XF32>(xg, dst, n, KCx, u);
            float sq = v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
            sq += __shfl_xor(sq, 1);
            sq += __shfl_xor(sq, 2);
            if (qd == 0 && dst >= 0) ssq[(size_t)dst * ssq_ld + grp] = sq;
        }
    }
};

// SwiGLU: packed rows alternate gate_j (2j) and up_j (2j+1); a = silu(gate) * up
// goes to the down projection's activation fragments (K = d_ff).
template <bool XF32>
struct EpiSwiGLU {
    void* a;
    int KCx;

    static constexpr int kSmem = 0;
    struct Pre {};
    __device__ void fetch(Pre&, int, int, int, int) const {}
    __device__ void stage(const Pre&, char*, int, int, int, int) const {}

    // four consecutive outputs (eight packed rows) per thread
    template <class SC>
    __device__ void operator()(float* Y, int ldy, int n0, int nrows, int m0, int mcols, int, char*,
                               const SC& sc) const {
        const int nq = nrows >> 3;
        for (int idx = threadIdx.x; idx < nq * mcols; idx += blockDim.x) {
            const int qd = idx % nq, ml = idx / nq;
            float v[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int ng = 8 * qd + 2 * e;
                const float gt = sc(Y[ng * ldy + ml], ng, ml), up = sc(Y[(ng + 1) * ldy + ml], ng + 1, ml);
                v[e] = gt / (1.0f + expf(-gt)) * up;
            }
            xfrag_store4<XF32>(a, m0 + ml, (n0 >> 1) + 4 * qd, KCx, make_float4(v[0], v[1], v[2], v[3]));
        }
    }
};

// LM head: per token, over this workgroup's vocabulary rows, the max logit, its
// lowest id and sum_v exp(l_v - max), MASK excluded; optionally the logits.
struct LmPartial {
    float mx;
    int arg;
    float s;
    float pad;
};

// Merge of two (max, lowest argmax, sum exp) records; symmetric in its operands.
__device__ __forceinline__ LmPartial lm_merge_fast(LmPartial a, LmPartial b) {
    if (b.arg < 0) return a;
    if (a.arg < 0) return b;
    const float mx = fmaxf(a.mx, b.mx);
    const int arg = (a.mx > b.mx) ? a.arg : (b.mx > a.mx ? b.arg : min(a.arg, b.arg));
    return LmPartial{mx, arg, a.s * __expf(a.mx - mx) + b.s * __expf(b.mx - mx), 0.f};
}

struct EpiLM {
    int V, mask_id, M;
    LmPartial* part;        // [n_groups][part_ld]
    int part_ld;
    float* logits;          // [M][V] or nullptr

    static constexpr int kSmem = 0;
    struct Pre {};
    __device__ void fetch(Pre&, int, int, int, int) const {}
    __device__ void stage(const Pre&, char*, int, int, int, int) const {}

    // TPT consecutive lanes per token, each an online (max, argmax, sum exp) over a
    // slice of the rows, then a fixed shuffle tree over the slices.
    template <class SC>
    __device__ void operator()(float* Y, int ldy, int n0, int nrows, int m0, int mcols, int grp, char*,
                               const SC& sc) const {
        if (logits != nullptr) {
            for (int idx = threadIdx.x; idx < nrows * mcols; idx += blockDim.x) {
                const int nl = idx % nrows, ml = idx / nrows;
                const int n = n0 + nl, m = m0 + ml;
                if (n < V && m < M)
                    logits[(size_t)m * V + n] = (n == mask_id) ? -INFINITY : sc(Y[nl * ldy + ml], nl, ml);
            }
        }
        // lanes per token: the largest power of two <= blockDim.x / mcols (groups of
        // tpt lanes are aligned inside a wave, so a group is wholly in or out of range)
        int tpt = 1;
        while (2 * tpt * mcols <= (int)blockDim.x && 2 * tpt <= 64) tpt *= 2;
        const int ml = threadIdx.x / tpt, sl = threadIdx.x % tpt;
        if (ml >= mcols) return;
        const int per = (nrows + tpt - 1) / tpt;
        const int b = sl * per, e = min(nrows, b + per);
        LmPartial a{-INFINITY, -1, 0.f, 0.f};
        for (int nl = b; nl < e; ++nl) {
            const int n = n0 + nl;
            if (n >= V || n == mask_id) continue;
            const float v = sc(Y[nl * ldy + ml], nl, ml);
            if (v > a.mx) {
                a.s = (a.arg < 0 ? 0.f : a.s * __expf(a.mx - v)) + 1.f;
                a.mx = v;
                a.arg = n;
            } else {
                a.s += __expf(v - a.mx);
            }
        }
        for (int off = 1; off < tpt; off <<= 1) {
            LmPartial o;
            o.mx = __shfl_xor(a.mx, off);
            o.arg = __shfl_xor(a.arg, off);
            o.s = __shfl_xor(a.s, off);
            o.pad = 0.f;
            a = lm_merge_fast(a, o);
        }
        if (sl == 0) part[(size_t)grp * part_ld + m0 + ml] = a;
    }
};

}  // namespace dllm
