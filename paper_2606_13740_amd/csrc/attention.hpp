// Window-vs-prefix attention (bidirectional inside the window, no causal mask).
//
// For a head h and a block of query rows, softmax(q k^T / sqrt(Dh)) v over keys
// [0, T) (or [0, lim[row]) for rows with their own limit), flash-style: the key
// range is cut into 32-key blocks; each wave streams its share of blocks with
// an online softmax; splits of the key range are merged by attn_combine.
//
// bf16 path on MFMA, computed transposed so that no operand needs a shuffle:
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
    const void* K;        // layer base [H][Cs][Dh]
    const void* Vt;       // layer base [H][Dh][Cs]
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

template <int DH, int QT>
__global__ void __launch_bounds__(64) attn_bf16_kernel(AttnArgs a) {
    constexpr int NC = DH / 32;     // 32-dim chunks
    constexpr int ND = DH / 16;     // 16-dim output tiles
    const int lane = threadIdx.x;
    const int r = lane & 15, g = lane >> 4;
    const int split = blockIdx.x, h = blockIdx.y;
    const int row0 = blockIdx.z * 16 * QT;
    const int ld = a.H * DH;
    const float sl2 = a.scale * 1.4426950408889634f;

    const uint16_t* qp = (const uint16_t*)a.q;
    const uint16_t* Kp = (const uint16_t*)a.K + (size_t)h * a.Cs * DH;
    const uint16_t* Vp = (const uint16_t*)a.Vt + (size_t)h * DH * a.Cs;

    u32x4_t qf[QT][NC];
    int lim[QT];
#pragma unroll
    for (int t = 0; t < QT; ++t) {
        const int row = row0 + 16 * t + r;
#pragma unroll
        for (int c = 0; c < NC; ++c) qf[t][c] = ldg16(qp + (size_t)row * ld + h * DH + 32 * c + 8 * g);
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

    const int nblk = (a.T + 31) >> 5;
    const int kb0 = split * a.bps;
    const int kb1 = min(nblk, kb0 + a.bps);
    const int krow0 = 8 * (r >> 2) + (r & 3);   // + 4t: the key this lane loads for tile t

    for (int kb = kb0; kb < kb1; ++kb) {
        const int k0 = kb * 32;
        u32x4_t kf[2][NC];
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int c = 0; c < NC; ++c)
                kf[t][c] = ldg16(Kp + (size_t)(k0 + krow0 + 4 * t) * DH + 32 * c + 8 * g);
        u32x4_t vf[ND];
#pragma unroll
        for (int dt = 0; dt < ND; ++dt) vf[dt] = ldg16(Vp + (size_t)(16 * dt + r) * a.Cs + k0 + 8 * g);
        if (k0 + 8 * g + 8 > a.T) {            // tail: zero V beyond T (the rows may be unwritten)
#pragma unroll
            for (int dt = 0; dt < ND; ++dt)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int key = k0 + 8 * g + 2 * e;
                    uint32_t w = vf[dt][e];
                    if (key >= a.T) w &= 0xFFFF0000u;
                    if (key + 1 >= a.T) w &= 0x0000FFFFu;
                    vf[dt][e] = w;
                }
        }

#pragma unroll
        for (int t = 0; t < QT; ++t) {
            f32x4_t s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                s0 = mfma_bf16(kf[0][c], qf[t][c], s0);
                s1 = mfma_bf16(kf[1][c], qf[t][c], s1);
            }
            float sv[8];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int key0 = k0 + 8 * g + i, key1 = key0 + 4;
                sv[i] = (key0 < lim[t]) ? s0[i] * sl2 : -INFINITY;
                sv[4 + i] = (key1 < lim[t]) ? s1[i] * sl2 : -INFINITY;
            }
            float bm = sv[0];
#pragma unroll
            for (int j = 1; j < 8; ++j) bm = fmaxf(bm, sv[j]);
            bm = fmaxf(bm, __shfl_xor(bm, 16));
            bm = fmaxf(bm, __shfl_xor(bm, 32));
            const float mnew = fmaxf(mrun[t], bm);
            float alpha = 1.f, ps = 0.f;
            uint32_t pk[4];
            if (mnew == -INFINITY) {
#pragma unroll
                for (int e = 0; e < 4; ++e) pk[e] = 0u;
            } else {
                alpha = exp2f(mrun[t] - mnew);
                float p[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) { p[j] = exp2f(sv[j] - mnew); ps += p[j]; }
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    pk[e] = (uint32_t)f32_to_bf16(p[2 * e]) | ((uint32_t)f32_to_bf16(p[2 * e + 1]) << 16);
            }
            lrun[t] = lrun[t] * alpha + ps;
            mrun[t] = mnew;
            const u32x4_t pf = {pk[0], pk[1], pk[2], pk[3]};
#pragma unroll
            for (int dt = 0; dt < ND; ++dt) {
#pragma unroll
                for (int i = 0; i < 4; ++i) oacc[dt][t][i] *= alpha;
                oacc[dt][t] = mfma_bf16(vf[dt], pf, oacc[dt][t]);
            }
        }
    }

#pragma unroll
    for (int t = 0; t < QT; ++t) {
        float l = lrun[t];
        l += __shfl_xor(l, 16);
        l += __shfl_xor(l, 32);
        const int row = row0 + 16 * t + r;
        if (a.nsplit == 1) {
            const float inv = 1.f / l;
#pragma unroll
            for (int dt = 0; dt < ND; ++dt)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    xfrag_store<false>(a.o, row, h * DH + 16 * dt + 4 * g + i, a.KCx, oacc[dt][t][i] * inv);
        } else {
            float* op = a.opart + (((size_t)split * a.rows_ld + row) * a.H + h) * DH;
#pragma unroll
            for (int dt = 0; dt < ND; ++dt)
#pragma unroll
                for (int i = 0; i < 4; ++i) op[16 * dt + 4 * g + i] = oacc[dt][t][i];
            if (g == 0) {
                float* ml = a.mlpart + (((size_t)split * a.rows_ld + row) * a.H + h) * 2;
                ml[0] = mrun[t];
                ml[1] = l;
            }
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
