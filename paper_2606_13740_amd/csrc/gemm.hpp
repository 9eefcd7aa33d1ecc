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
// Row scales (int8 weights) multiply Y per weight row; the RMSNorm factor
// rstd[m] of the consumer norm multiplies Y per token column: both factor out of
// the K sum, so the A operand only carries x * g (rounded once).
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
    // RMSNorm of the consumer: rstd[m] = 1 / sqrt(sum_p ssq[p][m] / d + eps)
    const float* ssq;     // [n_part][ssq_ld] partial sums of squares, or nullptr
    int n_part;
    int ssq_ld;
    float inv_d;
    float eps;
};

// Cooperative per-token 1/RMS from partial sums of squares, computed by one wave.
// Lane layout: G = mcols/4 float4 groups per partial row, nP = 64/G partial rows
// in flight per pass; partial sums are combined in LDS in a fixed order.
__device__ __forceinline__ void rstd_wave(const GemmArgs& g, int m0, int mcols, float* rstd_lds,
                                          float* tmp_lds /* >= 64 * 4 floats */) {
    const int lane = threadIdx.x & 63;
    const int G = mcols >> 2;
    const int nP = 64 / G;
    const int grp = lane % G, pr = lane / G;
    float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
    if (pr < nP) {
        const float* base = g.ssq + m0 + 4 * grp;
        int p = pr;
#pragma unroll 8
        for (; p < g.n_part; p += nP) {
            const float4 v = *(const float4*)(base + (size_t)p * g.ssq_ld);
            s0 += v.x; s1 += v.y; s2 += v.z; s3 += v.w;
        }
        tmp_lds[(pr * G + grp) * 4 + 0] = s0;
        tmp_lds[(pr * G + grp) * 4 + 1] = s1;
        tmp_lds[(pr * G + grp) * 4 + 2] = s2;
        tmp_lds[(pr * G + grp) * 4 + 3] = s3;
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (lane < mcols) {
        const int gg = lane >> 2, c = lane & 3;
        float t = 0.f;
        for (int q = 0; q < nP; ++q) t += tmp_lds[(q * G + gg) * 4 + c];
        rstd_lds[lane] = 1.0f / sqrtf(t * g.inv_d + g.eps);
    }
}

// Epilogue interface:  __device__ void operator()(const float* Y, int ldy, int n0, int nrows,
//                                                 int m0, int mcols, float* scratch) const
// Y is LDS [nrows][ldy] holding final outputs (scales and rstd applied); all
// threads of the workgroup call it; scratch is LDS of at least nrows*ldy floats
// that the epilogue may overwrite (it aliases Y).

// Loads in flight per wave: as many K chunks as fit in ~128 VGPRs of buffers.
template <int WT, int F, int MT>
constexpr int pipeline_depth() {
    constexpr int XP = (WT == WT_F32) ? 1 : 2;
    constexpr int slot = 4 * (F + MT * WTraits<WT>::XPER * XP);
    constexpr int d = 128 / slot;
    return d < 1 ? 1 : (d > 8 ? 8 : d);
}

template <int WT, int F, int MT, int NW, bool RSTD, class Epi>
__global__ void __launch_bounds__((NW + (RSTD ? 1 : 0)) * 64)
gemm_kernel(GemmArgs g, Epi epi) {
    constexpr int XPER = WTraits<WT>::XPER;
    constexpr bool XF = (WT == WT_F32);
    constexpr int XP = XF ? 1 : 2;                 // activation planes (hi, lo)
    constexpr int XB = XChunk<XF>::bytes;
    constexpr int D = pipeline_depth<WT, F, MT>();
    constexpr int NR = 16 * F, MR = 16 * MT, LDY = MR + 1;
    __shared__ float Y[NR * LDY];
    __shared__ float rstd_lds[64];
    __shared__ float tmp_lds[64 * 4];

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int nt0 = blockIdx.x * F;
    const int mt0 = blockIdx.y * MT;
    const int nf = min(F, g.n_tiles - nt0);  // valid row tiles of this workgroup

    f32x4_t acc[F][MT];
#pragma unroll
    for (int f = 0; f < F; ++f)
#pragma unroll
        for (int t = 0; t < MT; ++t) acc[f][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    if (wave < NW) {
        const int c0 = (int)(((long)wave * g.KCw) / NW);
        const int c1 = (int)(((long)(wave + 1) * g.KCw) / NW);
        const char* wp = (const char*)g.W + ((size_t)nt0 * g.KCw * 64 + lane) * 16;
        const char* xp = (const char*)g.X + (size_t)mt0 * g.KCx * XB + lane * 16;
        const size_t wtile = (size_t)g.KCw * 1024, xtile = (size_t)g.KCx * XB;

        u32x4_t wb[D][F];
        u32x4_t xb[D][MT * XPER * XP];

        auto load = [&](int s, int c) {
#pragma unroll
            for (int f = 0; f < F; ++f)
                if (f < nf) wb[s][f] = ldg16_nt(wp + f * wtile + (size_t)c * 1024);
#pragma unroll
            for (int t = 0; t < MT; ++t)
#pragma unroll
                for (int h = 0; h < XPER; ++h)
#pragma unroll
                    for (int pl = 0; pl < XP; ++pl)
                        xb[s][(t * XPER + h) * XP + pl] =
                            ldg16(xp + t * xtile + (size_t)(c * XPER + h) * XB + pl * 1024);
        };
        auto compute = [&](int s) {
#pragma unroll
            for (int f = 0; f < F; ++f) {
                if (f >= nf) continue;
                if constexpr (WT == WT_BF16) {
#pragma unroll
                    for (int t = 0; t < MT; ++t) {
                        acc[f][t] = mfma_bf16(wb[s][f], xb[s][t * 2 + 0], acc[f][t]);
                        acc[f][t] = mfma_bf16(wb[s][f], xb[s][t * 2 + 1], acc[f][t]);
                    }
                } else if constexpr (WT == WT_I8) {
                    const u32x4_t w0 = i8x8_to_bf16x8(wb[s][f][0], wb[s][f][1]);
                    const u32x4_t w1 = i8x8_to_bf16x8(wb[s][f][2], wb[s][f][3]);
#pragma unroll
                    for (int t = 0; t < MT; ++t) {
                        acc[f][t] = mfma_bf16(w0, xb[s][(t * 2 + 0) * 2 + 0], acc[f][t]);
                        acc[f][t] = mfma_bf16(w0, xb[s][(t * 2 + 0) * 2 + 1], acc[f][t]);
                        acc[f][t] = mfma_bf16(w1, xb[s][(t * 2 + 1) * 2 + 0], acc[f][t]);
                        acc[f][t] = mfma_bf16(w1, xb[s][(t * 2 + 1) * 2 + 1], acc[f][t]);
                    }
                } else {
#pragma unroll
                    for (int t = 0; t < MT; ++t)
#pragma unroll
                        for (int q = 0; q < 4; ++q)
                            acc[f][t] = mfma_f32(__uint_as_float(wb[s][f][q]), __uint_as_float(xb[s][t][q]),
                                                 acc[f][t]);
                }
            }
        };

        if (c1 > c0) {
#pragma unroll
            for (int s = 0; s < D; ++s) load(s, min(c0 + s, c1 - 1));
            for (int base = c0; base < c1; base += D) {
#pragma unroll
                for (int s = 0; s < D; ++s) {
                    const int c = base + s;
                    if (c < c1) compute(s);
                    const int cn = c + D;
                    if (cn < c1) load(s, cn);
                }
            }
        }
    } else if constexpr (RSTD) {
        rstd_wave(g, mt0 * 16, MR, rstd_lds, tmp_lds);
    }

    // Combine the NW partial tiles in LDS, wave by wave (fixed order).
    const int r = lane & 15, gq = lane >> 4;
    for (int w = 0; w < NW; ++w) {
        if (wave == w) {
#pragma unroll
            for (int f = 0; f < F; ++f)
#pragma unroll
                for (int t = 0; t < MT; ++t)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        float* p = &Y[(16 * f + 4 * gq + i) * LDY + 16 * t + r];
                        *p = (w == 0) ? acc[f][t][i] : *p + acc[f][t][i];
                    }
        }
        __syncthreads();
    }

    // Row scales and per-token rstd.
    if (g.wscale != nullptr || RSTD) {
        for (int idx = threadIdx.x; idx < NR * MR; idx += blockDim.x) {
            const int n = idx / MR, m = idx % MR;
            float v = Y[n * LDY + m];
            if (g.wscale != nullptr) {
                const int gn = nt0 * 16 + n;
                v *= (gn < g.n_tiles * 16) ? g.wscale[gn] : 0.f;
            }
            if constexpr (RSTD) v *= rstd_lds[m];
            Y[n * LDY + m] = v;
        }
        __syncthreads();
    }
    epi(Y, LDY, nt0 * 16, nf * 16, mt0 * 16, MR);
}

// ---------------------------------------------------------------------------
// Epilogues
// ---------------------------------------------------------------------------

// Q/K/V projection: RoPE on Q and K, Q to a row-major buffer, K and V to the
// cache at each token's position.  Packed rows: [Q | K | V], each d rows; inside
// a Q or K head, packed row 2i is dim i and row 2i+1 is dim i + Dh/2, so a RoPE
// pair is two adjacent rows.  fp32 models store one fp32 plane; bf16 / int8
// models store a hi and a lo bf16 plane (`plane` elements apart).
template <bool XF32>
struct EpiQKV {
    using T = typename std::conditional<XF32, float, uint16_t>::type;
    int d, Dh, M;
    int pos_base;           // position of token m is pos ? pos[m] : pos_base + m
    const int* pos;
    const float2* rope;     // [max_pos][Dh/2] (cos, sin)
    T* q;                   // [rows][d] (+ lo plane at q + q_plane)
    size_t q_plane;
    T* Kc;                  // layer base of K   [H][Cs][Dh] (+ lo plane at kv_plane)
    T* Vt;                  // layer base of V^T [H][Dh][Cs] (+ lo plane at kv_plane)
    size_t kv_plane;
    int Cs;

    __device__ __forceinline__ static void put(T* p, size_t plane, float v) {
        if constexpr (XF32) {
            *p = v;
        } else {
            uint16_t hi, lo;
            split_bf16(v, hi, lo);
            p[0] = hi;
            p[plane] = lo;
        }
    }

    __device__ void operator()(const float* Y, int ldy, int n0, int nrows, int m0, int mcols) const {
        const int npairs = nrows >> 1;
        const int half = Dh >> 1;
        for (int idx = threadIdx.x; idx < npairs * mcols; idx += blockDim.x) {
            const int p = idx % npairs, ml = idx / npairs;
            const int m = m0 + ml;
            if (m >= M) continue;
            const int n = n0 + 2 * p;
            const float a = Y[(2 * p) * ldy + ml], b = Y[(2 * p + 1) * ldy + ml];
            const int ps = pos ? pos[m] : pos_base + m;
            const int seg = n / d, nn = n - seg * d;
            const int h = nn / Dh, rr = nn - h * Dh;
            if (seg < 2) {
                const int j = rr >> 1;
                const float2 cs = rope[(size_t)ps * half + j];
                const float ra = a * cs.x - b * cs.y;
                const float rb = a * cs.y + b * cs.x;
                if (seg == 0) {
                    T* dst = q + (size_t)m * d + h * Dh;
                    put(dst + j, q_plane, ra);
                    put(dst + j + half, q_plane, rb);
                } else {
                    T* dst = Kc + ((size_t)h * Cs + ps) * Dh;
                    put(dst + j, kv_plane, ra);
                    put(dst + j + half, kv_plane, rb);
                }
            } else {
                T* dst = Vt + ((size_t)h * Dh + rr) * Cs + ps;
                put(dst, kv_plane, a);
                put(dst + Cs, kv_plane, b);
            }
        }
    }
};

// x += Y^T (residual), then the next RMSNorm's A operand xg = bf16(x * g_next)
// and this workgroup's partial sum of squares of x per token.
template <bool XF32>
struct EpiResidual {
    float* x;               // [rows][d]
    int d, M;
    const float* gnext;     // [d]
    void* xg;               // activation fragments, K = d
    int KCx;
    float* ssq;             // [n_part][ssq_ld]
    int ssq_ld;

    __device__ void operator()(float* Y, int ldy, int n0, int nrows, int m0, int mcols) const {
        for (int idx = threadIdx.x; idx < nrows * mcols; idx += blockDim.x) {
            const int nl = idx % nrows, ml = idx / nrows;
            const int m = m0 + ml, n = n0 + nl;
            float sq = 0.f;
            if (m < M) {
                float* xp = x + (size_t)m * d + n;
                const float xv = *xp + Y[nl * ldy + ml];
                *xp = xv;
                xfrag_store<XF32>(xg, m, n, KCx, xv * gnext[n]);
                sq = xv * xv;
            } else {
                xfrag_store<XF32>(xg, m, n, KCx, 0.f);
            }
            Y[nl * ldy + ml] = sq;
        }
        __syncthreads();
        for (int ml = threadIdx.x; ml < mcols; ml += blockDim.x) {
            float s = 0.f;
            for (int nl = 0; nl < nrows; ++nl) s += Y[nl * ldy + ml];
            ssq[(size_t)blockIdx.x * ssq_ld + m0 + ml] = s;
        }
    }
};

// SwiGLU: packed rows alternate gate_j (2j) and up_j (2j+1); a = silu(gate) * up
// goes to the down projection's activation fragments (K = d_ff).
template <bool XF32>
struct EpiSwiGLU {
    void* a;
    int KCx;

    __device__ void operator()(const float* Y, int ldy, int n0, int nrows, int m0, int mcols) const {
        const int npairs = nrows >> 1;
        for (int idx = threadIdx.x; idx < npairs * mcols; idx += blockDim.x) {
            const int p = idx % npairs, ml = idx / npairs;
            const float gt = Y[(2 * p) * ldy + ml], up = Y[(2 * p + 1) * ldy + ml];
            const float act = gt / (1.0f + expf(-gt)) * up;
            xfrag_store<XF32>(a, m0 + ml, (n0 >> 1) + p, KCx, act);
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

struct EpiLM {
    int V, mask_id, M;
    LmPartial* part;        // [n_wg][part_ld]
    int part_ld;
    float* logits;          // [M][V] or nullptr

    __device__ void operator()(const float* Y, int ldy, int n0, int nrows, int m0, int mcols) const {
        if (logits != nullptr) {
            for (int idx = threadIdx.x; idx < nrows * mcols; idx += blockDim.x) {
                const int nl = idx % nrows, ml = idx / nrows;
                const int n = n0 + nl, m = m0 + ml;
                if (n < V && m < M)
                    logits[(size_t)m * V + n] = (n == mask_id) ? -INFINITY : Y[nl * ldy + ml];
            }
        }
        for (int ml = threadIdx.x; ml < mcols; ml += blockDim.x) {
            float mx = -INFINITY;
            int arg = -1;
            for (int nl = 0; nl < nrows; ++nl) {
                const int n = n0 + nl;
                if (n >= V || n == mask_id) continue;
                const float v = Y[nl * ldy + ml];
                if (v > mx) { mx = v; arg = n; }
            }
            float s = 0.f;
            if (arg >= 0) {
                for (int nl = 0; nl < nrows; ++nl) {
                    const int n = n0 + nl;
                    if (n >= V || n == mask_id) continue;
                    s += expf(Y[nl * ldy + ml] - mx);
                }
            }
            part[(size_t)blockIdx.x * part_ld + m0 + ml] = LmPartial{mx, arg, s, 0.f};
        }
    }
};

}  // namespace dllm
