// Window-vs-prefix attention (bidirectional inside the window, no causal mask).
//
// For a head h and a block of query rows, softmax(q k^T / sqrt(Dh)) v over keys
// [0, T) (or [0, lim[row]) for rows with their own limit), flash-style: the key
// range is cut into 32-key blocks; each wave streams its share of blocks with
// an online softmax; splits of the key range are merged by attn_combine.
//
// MFMA path, computed transposed so that no operand needs a shuffle:
//   S^T (16 keys x 16 queries) = K_tile (A: 16 keys x 32 dims) * Q^T (B)
//   O^T (16 dims x 16 queries) += V^T_tile (A: 16 dims x 32 keys) * P^T (B)
// K rows are loaded in the order key = 8*(r/4) + 4t + r%4 for tile t, so that
// lane group g ends up holding the probabilities of keys 8g .. 8g+7 of the
// block in B-operand order, and V^T (stored [dim][pos]) gives those 8 keys as
// one 16-byte load.
#pragma once

#include "common.hpp"

namespace dllm {

struct AttnArgs {
    const void* q;        // [rows][H][Dh]
    size_t q_plane;       // elements from the hi to the lo plane of q (bf16 path)
    const void* K;        // layer base [H][Cs][Dh]
    const void* Vt;       // layer base [H][Dh][Cs]
    size_t kv_plane;      // elements from the hi to the lo plane of K and V^T (bf16 path)
    int Cs;               // cache row stride (multiple of 32)
    int H;
    int T;                // keys [0, T) for rows without their own limit
    const int* lim;       // per-row key limit (rows < M) or nullptr
    int M;                // real rows
    int nsplit, bps;      // key-range splits, 32-key blocks per split
    float scale;          // 1 / sqrt(Dh)
    void* o;              // output fragments (K = d), used when nsplit == 1
    int KCx;
    float* opart;         // [nsplit][rows_ld][H][Dh]  unnormalised partial outputs
    float* mlpart;        // [nsplit][rows_ld][H][2]   (running max in log2 units, sum)
    int rows_ld;
};

// bf16 MFMA path.  Q, K and V are carried as hi + lo bf16 planes and each
// product takes three MFMAs (hi*hi + hi*lo + lo*hi), so scores and outputs keep
// ~16 significant bits; the probabilities P are split the same way.
//
// Workgroup = (split, head, query block of 16*QT rows) with NWA waves; the
// split's 32-key blocks are dealt out to the waves in contiguous runs, each
// wave keeps its own online softmax, and the waves are merged in LDS (max over
// waves, then the rescaled outputs summed wave by wave in a fixed order).  With
// one split the normalised output goes straight to the O projection's
// fragments; otherwise (m, l, o) per split goes to attn_combine.
template <int DH, int QT, int NWA>
__global__ void __launch_bounds__(NWA * 64) attn_bf16_kernel(AttnArgs a) {
    constexpr int NC = DH / 32;     // 32-dim chunks
    constexpr int ND = DH / 16;     // 16-dim output tiles
    constexpr int NQ = 16 * QT;     // query rows of the workgroup
    __shared__ float mx_s[NWA][NQ];
    __shared__ float l_s[NWA][NQ];
    __shared__ float obuf[NQ][DH + 1];
    __shared__ float Mq[NQ], Lq[NQ];

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int split = blockIdx.x, h = blockIdx.y;
    const int row0 = blockIdx.z * NQ;
    const int ld = a.H * DH;
    const float sl2 = a.scale * 1.4426950408889634f;

    const uint16_t* qp = (const uint16_t*)a.q;
    const uint16_t* Kp = (const uint16_t*)a.K + (size_t)h * a.Cs * DH;
    const uint16_t* Vp = (const uint16_t*)a.Vt + (size_t)h * DH * a.Cs;

    const int nblk = (a.T + 31) >> 5;
    const int sb0 = split * a.bps, sb1 = min(nblk, sb0 + a.bps);
    const int kb0 = sb0 + (int)(((long)wave * (sb1 - sb0)) / NWA);
    const int kb1 = sb0 + (int)(((long)(wave + 1) * (sb1 - sb0)) / NWA);

    u32x4_t qf[QT][NC][2];
    int lim[QT];
#pragma unroll
    for (int t = 0; t < QT; ++t) {
        const int row = row0 + 16 * t + r;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const uint16_t* src = qp + (size_t)row * ld + h * DH + 32 * c + 8 * g;
            qf[t][c][0] = ldg16(src);
            qf[t][c][1] = ldg16(src + a.q_plane);
        }
        lim[t] = (a.lim != nullptr && row < a.M) ? a.lim[row] : a.T;
    }

    float mrun[QT], lrun[QT];
    f32x4_t oacc[ND][QT];
#pragma unroll
    for (int t = 0; t < QT; ++t) {
        mrun[t] = -INFINITY;
        lrun[t] = 0.f;
#pragma unroll
        for (int dt = 0; dt < ND; ++dt) oacc[dt][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }

    const int krow0 = 8 * (r >> 2) + (r & 3);   // + 4t: the key this lane loads for tile t

    for (int kb = kb0; kb < kb1; ++kb) {
        const int k0 = kb * 32;
        // issue the block's K and V loads together
        u32x4_t kf[NC][2][2];
#pragma unroll
        for (int c = 0; c < NC; ++c)
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                const uint16_t* src = Kp + (size_t)(k0 + krow0 + 4 * t) * DH + 32 * c + 8 * g;
                kf[c][t][0] = ldg16(src);
                kf[c][t][1] = ldg16(src + a.kv_plane);
            }
        u32x4_t vf[ND][2];
#pragma unroll
        for (int dt = 0; dt < ND; ++dt) {
            const uint16_t* src = Vp + (size_t)(16 * dt + r) * a.Cs + k0 + 8 * g;
            vf[dt][0] = ldg16(src);
            vf[dt][1] = ldg16(src + a.kv_plane);
        }

        // scores S^T for both 16-key tiles and every query tile
        f32x4_t sacc[2][QT];
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int u = 0; u < QT; ++u) sacc[t][u] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < NC; ++c)
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int u = 0; u < QT; ++u) {
                    sacc[t][u] = mfma_bf16(kf[c][t][0], qf[u][c][0], sacc[t][u]);
                    sacc[t][u] = mfma_bf16(kf[c][t][0], qf[u][c][1], sacc[t][u]);
                    sacc[t][u] = mfma_bf16(kf[c][t][1], qf[u][c][0], sacc[t][u]);
                }

        u32x4_t pf[QT][2];
#pragma unroll
        for (int u = 0; u < QT; ++u) {
            float sv[8];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int key0 = k0 + 8 * g + i, key1 = key0 + 4;
                sv[i] = (key0 < lim[u]) ? sacc[0][u][i] * sl2 : -INFINITY;
                sv[4 + i] = (key1 < lim[u]) ? sacc[1][u][i] * sl2 : -INFINITY;
            }
            float bm = sv[0];
#pragma unroll
            for (int j = 1; j < 8; ++j) bm = fmaxf(bm, sv[j]);
            bm = fmaxf(bm, __shfl_xor(bm, 16));
            bm = fmaxf(bm, __shfl_xor(bm, 32));
            const float mnew = fmaxf(mrun[u], bm);
            float alpha = 1.f, ps = 0.f;
            uint32_t phi[4] = {0u, 0u, 0u, 0u}, plo[4] = {0u, 0u, 0u, 0u};
            if (mnew != -INFINITY) {
                alpha = exp2f(mrun[u] - mnew);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float p0 = exp2f(sv[2 * e] - mnew), p1 = exp2f(sv[2 * e + 1] - mnew);
                    ps += p0 + p1;
                    uint16_t h0, l0, h1, l1;
                    split_bf16(p0, h0, l0);
                    split_bf16(p1, h1, l1);
                    phi[e] = (uint32_t)h0 | ((uint32_t)h1 << 16);
                    plo[e] = (uint32_t)l0 | ((uint32_t)l1 << 16);
                }
            }
            lrun[u] = lrun[u] * alpha + ps;
            mrun[u] = mnew;
            pf[u][0] = u32x4_t{phi[0], phi[1], phi[2], phi[3]};
            pf[u][1] = u32x4_t{plo[0], plo[1], plo[2], plo[3]};
#pragma unroll
            for (int dt = 0; dt < ND; ++dt)
#pragma unroll
                for (int i = 0; i < 4; ++i) oacc[dt][u][i] *= alpha;
        }

        // O^T += V^T * P^T
        if (k0 + 8 * g + 8 > a.T) {            // tail: zero V beyond T (those rows may be unwritten)
#pragma unroll
            for (int dt = 0; dt < ND; ++dt)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int key = k0 + 8 * g + 2 * e;
                    const uint32_t keep = (key >= a.T ? 0u : 0x0000FFFFu) | (key + 1 >= a.T ? 0u : 0xFFFF0000u);
                    vf[dt][0][e] &= keep;
                    vf[dt][1][e] &= keep;
                }
        }
#pragma unroll
        for (int dt = 0; dt < ND; ++dt)
#pragma unroll
            for (int u = 0; u < QT; ++u) {
                oacc[dt][u] = mfma_bf16(vf[dt][0], pf[u][0], oacc[dt][u]);
                oacc[dt][u] = mfma_bf16(vf[dt][0], pf[u][1], oacc[dt][u]);
                oacc[dt][u] = mfma_bf16(vf[dt][1], pf[u][0], oacc[dt][u]);
            }
    }

    // ---- merge the NWA waves ----
#pragma unroll
    for (int u = 0; u < QT; ++u) {
        float l = lrun[u];
        l += __shfl_xor(l, 16);
        l += __shfl_xor(l, 32);
        if (g == 0) {
            mx_s[wave][16 * u + r] = mrun[u];
            l_s[wave][16 * u + r] = l;
        }
    }
    __syncthreads();
    for (int q = threadIdx.x; q < NQ; q += blockDim.x) {
        float M = -INFINITY;
        for (int w = 0; w < NWA; ++w) M = fmaxf(M, mx_s[w][q]);
        float L = 0.f;
        for (int w = 0; w < NWA; ++w)
            if (mx_s[w][q] != -INFINITY) L += l_s[w][q] * exp2f(mx_s[w][q] - M);
        Mq[q] = M;
        Lq[q] = L;
    }
    __syncthreads();
    for (int w = 0; w < NWA; ++w) {
        if (wave == w) {
#pragma unroll
            for (int u = 0; u < QT; ++u) {
                const int q = 16 * u + r;
                const float sc = (mrun[u] == -INFINITY) ? 0.f : exp2f(mrun[u] - Mq[q]);
#pragma unroll
                for (int dt = 0; dt < ND; ++dt)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        float* o = &obuf[q][16 * dt + 4 * g + i];
                        *o = (w == 0 ? 0.f : *o) + oacc[dt][u][i] * sc;
                    }
            }
        }
        __syncthreads();
    }
    if (a.nsplit == 1) {
        for (int idx = threadIdx.x; idx < NQ * DH; idx += blockDim.x) {
            const int q = idx / DH, dim = idx % DH;
            xfrag_store<false>(a.o, row0 + q, h * DH + dim, a.KCx, obuf[q][dim] / Lq[q]);
        }
    } else {
        for (int idx = threadIdx.x; idx < NQ * DH; idx += blockDim.x) {
            const int q = idx / DH, dim = idx % DH;
            a.opart[(((size_t)split * a.rows_ld + row0 + q) * a.H + h) * DH + dim] = obuf[q][dim];
        }
        for (int q = threadIdx.x; q < NQ; q += blockDim.x) {
            float* ml = a.mlpart + (((size_t)split * a.rows_ld + row0 + q) * a.H + h) * 2;
            ml[0] = Mq[q];
            ml[1] = Lq[q];
        }
    }
}

// Merge key-range splits: O = sum_s o_s 2^(m_s - M) / sum_s l_s 2^(m_s - M).
template <bool XF32>
__global__ void __launch_bounds__(256) attn_combine_kernel(AttnArgs a, int rows, int DH) {
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    const int total = rows * a.H * DH;
    if (idx >= total) return;
    const int dim = idx % DH;
    const int h = (idx / DH) % a.H;
    const int row = idx / (DH * a.H);
    float mx = -INFINITY;
    for (int s = 0; s < a.nsplit; ++s)
        mx = fmaxf(mx, a.mlpart[(((size_t)s * a.rows_ld + row) * a.H + h) * 2]);
    float l = 0.f, o = 0.f;
    for (int s = 0; s < a.nsplit; ++s) {
        const float* ml = a.mlpart + (((size_t)s * a.rows_ld + row) * a.H + h) * 2;
        if (ml[0] == -INFINITY) continue;
        const float w = exp2f(ml[0] - mx);
        l += ml[1] * w;
        o += a.opart[(((size_t)s * a.rows_ld + row) * a.H + h) * DH + dim] * w;
    }
    xfrag_store<XF32>(a.o, row, h * DH + dim, a.KCx, o / l);
}

// fp32 path (small models): one wave per (row, head); lanes stride over keys with
// a lane-local online softmax, merged across lanes by a butterfly.
template <int DH>
__global__ void __launch_bounds__(64) attn_f32_kernel(AttnArgs a) {
    const int lane = threadIdx.x;
    const int row = blockIdx.x, h = blockIdx.y;
    const int ld = a.H * DH;
    const float* qp = (const float*)a.q + (size_t)row * ld + h * DH;
    const float* Kp = (const float*)a.K + (size_t)h * a.Cs * DH;
    const float* Vp = (const float*)a.Vt + (size_t)h * DH * a.Cs;
    const int lim = (a.lim != nullptr && row < a.M) ? a.lim[row] : a.T;

    float q[DH];
#pragma unroll
    for (int j = 0; j < DH; ++j) q[j] = qp[j];
    float m = -INFINITY, l = 0.f;
    float o[DH];
#pragma unroll
    for (int j = 0; j < DH; ++j) o[j] = 0.f;
    for (int k = lane; k < lim; k += 64) {
        const float* kr = Kp + (size_t)k * DH;
        float s = 0.f;
#pragma unroll
        for (int j = 0; j < DH; ++j) s = fmaf(q[j], kr[j], s);
        s *= a.scale;
        const float mn = fmaxf(m, s);
        const float alpha = expf(m - mn);
        const float p = expf(s - mn);
        l = l * alpha + p;
#pragma unroll
        for (int j = 0; j < DH; ++j) o[j] = o[j] * alpha + p * Vp[(size_t)j * a.Cs + k];
        m = mn;
    }
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const float m2 = __shfl_xor(m, off), l2 = __shfl_xor(l, off);
        const float mn = fmaxf(m, m2);
        const float w1 = (m == -INFINITY) ? 0.f : expf(m - mn);
        const float w2 = (m2 == -INFINITY) ? 0.f : expf(m2 - mn);
        l = l * w1 + l2 * w2;
#pragma unroll
        for (int j = 0; j < DH; ++j) o[j] = o[j] * w1 + __shfl_xor(o[j], off) * w2;
        m = mn;
    }
    const float inv = 1.f / l;
#pragma unroll
    for (int j = 0; j < DH; ++j)
        if ((j & 63) == lane) xfrag_store<true>(a.o, row, h * DH + j, a.KCx, o[j] * inv);
}

}  // namespace dllm
