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
    size_t q_plane;       // elements from the hi to the lo plane of q (fp16 path)
    const void* K;        // layer base [Hkv][Cs][Dh]
    const void* Vt;       // layer base [Hkv][Dh][Cs]
    int Cs;               // cache row stride (multiple of 32)
    int H;                // query heads
    int G;                // query heads per K/V head (grouped-query attention; 1 = multi-head)
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

// fp16 MFMA path (v_mfma_f32_16x16x32_f16).  The cache holds K and V^T as one fp16
// plane each; Q arrives as an fp16 hi + lo pair and the probabilities P are split the
// same way in registers, so every product takes two MFMAs (K * Q_hi + K * Q_lo,
// V^T * P_hi + V^T * P_lo) and the scores and outputs keep the cache's precision.
//
// Workgroup = (key split, head, group of QG query tiles of 16 rows), KS x QG waves:
// KS key groups of QG waves, one wave per query tile.  Key group k takes the split's
// 32-key blocks k, k + KS, ...; each block is staged in the group's own LDS buffers
// once with direct global->LDS loads (global_load_lds_dwordx4) in a ring of NB buffers,
// so the next NB - 1 blocks stream in while the current one is used, and the group's waves read
// their MFMA fragments from LDS.  With KS > 1 the groups' partial (max, sum, O)
// states are merged in LDS in group order at the end.  LDS rows are XOR-swizzled in 16-byte columns so that
// the 16 rows one fragment read touches fall in distinct banks:
//   K  [32 keys][Dh/8 cols]: col' = col ^ (((key & 3) | (4 * ((key >> 3) & 3))) mod Dh/8)
//   V^T [Dh dims][4 cols]:   col' = col ^ ((dim >> 2) & 3)
// With one split the normalised output goes to the O projection's fragments;
// otherwise (m, l, o) per split goes to attn_combine.  Short key ranges take KS > 1
// and a single split, which leaves no merge launch.
__device__ __forceinline__ int swz_k(int key) { return (key & 3) | (((key >> 3) & 3) << 2); }

typedef __attribute__((address_space(3))) void lds_void;

// At most two waves per SIMD's worth of registers (256): with the 512 a workgroup of
// 2-4 waves may take, the compiler chose the AGPR form of the MFMAs and copied every
// output tile VGPR -> AGPR around each product.
// Staging buffers per workgroup with one key group (KS = 1).
constexpr int ATTN_RING = 2;
// log2-domain slack of the lazily rescaled softmax maximum: probabilities <= 2^8
constexpr float ATTN_SLACK = 8.f;

template <int DH, int QG, int KS, int NB>
__global__ void __launch_bounds__(QG * KS * 64) __attribute__((amdgpu_waves_per_eu(2)))
attn_f16_kernel(AttnArgs a) {
    constexpr int NC = DH / 32;               // 32-dim chunks
    constexpr int ND = DH / 16;               // 16-dim output tiles
    constexpr int KCOLS = DH / 8;             // 16-byte columns per key row
    constexpr int KPLANE = 32 * DH * 2;       // bytes of a block's K (fp16)
    constexpr int VPLANE = DH * 64;           // bytes of a block's V^T (fp16)
    constexpr int BUF = KPLANE + VPLANE;
    constexpr int NSLOT = BUF / 16;           // 16-byte slots per block
    static_assert(NSLOT % 64 == 0, "block must be whole wave loads");
    constexpr int MLD = DH + 4;               // merge: floats per (group, row) record
    constexpr int MERGE = KS > 1 ? KS * QG * 16 * (MLD + 2) * 4 : 0;
    static_assert(NB >= 2 && NB <= 4, "2-4 staging buffers per key group");
    constexpr int LPW = (NSLOT / 64) / QG;    // loads each wave issues per staged block, at least
    __shared__ __attribute__((aligned(1024))) char lds[KS * NB * BUF > MERGE ? KS * NB * BUF : MERGE];

    const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int r = lane & 15, g = lane >> 4;
    const int grp = wave / QG, qw = wave % QG;                // key group, query tile
    // 1-D grid over (head h, query group z, split) items, in that order.  The dispatcher
    // deals consecutive workgroups to the 8 XCDs in turn; when the items divide into
    // 8 equal shares, XCD x takes the x-th share, so the query groups and splits of a
    // head (which read the same K/V, the splits adjacent 64-byte halves of the same
    // V^T lines) share one L2.
    const int nitems = (int)gridDim.x;
    const int nqg = nitems / (a.nsplit * a.H);
    int item = blockIdx.x;
    if ((nitems & 7) == 0) item = (blockIdx.x & 7) * (nitems >> 3) + (blockIdx.x >> 3);
    const int split = item % a.nsplit, z = (item / a.nsplit) % nqg, h = item / (a.nsplit * nqg);
    const int row = z * 16 * QG + 16 * qw + r;               // this lane's query row
    const int ld = a.H * DH;
    const float sl2 = a.scale * 1.4426950408889634f;

    const uint16_t* qp = (const uint16_t*)a.q;
    const int hk = h / a.G;                                  // K/V head of this query head
    const uint16_t* Kp = (const uint16_t*)a.K + (size_t)hk * a.Cs * DH;
    const uint16_t* Vp = (const uint16_t*)a.Vt + (size_t)hk * DH * a.Cs;

    const int nblk = (a.T + 31) >> 5;
    const int kb0 = split * a.bps, kb1 = min(nblk, kb0 + a.bps);

    // stage block kb into the group's buffer `buf`: slot s -> K plane / V^T plane position
    auto stage = [&](int kb, int buf) {
        const int k0 = kb * 32;
        char* base = lds + (grp * NB + buf) * BUF;
#pragma unroll
        for (int j = 0; j < (NSLOT / 64 + QG - 1) / QG; ++j) {
            const int i = qw + j * QG;
            if (i >= NSLOT / 64) break;
            const int sl = i * 64 + lane;
            const uint16_t* src;
            if (sl < KPLANE / 16) {                      // K: 32 x KCOLS slots
                const int key = sl / KCOLS, pc = sl % KCOLS;
                const int col = pc ^ (swz_k(key) & (KCOLS - 1));
                src = Kp + (size_t)(k0 + key) * DH + col * 8;
            } else {                                     // V^T: DH x 4 slots
                const int s1 = sl - KPLANE / 16;
                const int dim = s1 >> 2, pc = s1 & 3;
                const int col = pc ^ ((dim >> 2) & 3);
                src = Vp + (size_t)dim * a.Cs + k0 + col * 8;
            }
            __builtin_amdgcn_global_load_lds((const void*)src, (lds_void*)(base + i * 1024), 16, 0, 0);
        }
    };

    // zero the V^T values of keys >= T in the slots this wave staged into buffer `buf`
    // (cache rows past T may hold anything, and 0 * NaN would reach O); K needs no
    // such care, its scores past T are masked
    auto zero_tail = [&](int kb, int buf) {
        const int k0 = kb * 32;
        char* base = lds + (grp * NB + buf) * BUF;
#pragma unroll
        for (int j = 0; j < (NSLOT / 64 + QG - 1) / QG; ++j) {
            const int i = qw + j * QG;
            if (i >= NSLOT / 64) break;
            const int sl = i * 64 + lane;
            if (sl < KPLANE / 16) continue;
            const int s1 = sl - KPLANE / 16;
            const int dim = s1 >> 2, pc = s1 & 3;
            const int key = k0 + 8 * (pc ^ ((dim >> 2) & 3));      // the slot's first key
            if (key + 8 <= a.T) continue;
            u32x4_t* slot = (u32x4_t*)(base + i * 1024 + lane * 16);
            u32x4_t v = *slot;
#pragma unroll
            for (int e = 0; e < 4; ++e)
                v[e] &= (key + 2 * e >= a.T ? 0u : 0x0000FFFFu) | (key + 2 * e + 1 >= a.T ? 0u : 0xFFFF0000u);
            *slot = v;
        }
    };

    u32x4_t qf[NC][2];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const uint16_t* src = qp + (size_t)row * ld + h * DH + 32 * c + 8 * g;
        qf[c][0] = ldg16(src);
        qf[c][1] = ldg16(src + a.q_plane);
    }
    const int lim = (a.lim != nullptr && row < a.M) ? a.lim[row] : a.T;

    // Ring of NB buffers per key group: the group's first NB - 1 blocks are staged
    // here (after the Q loads, so the ring's waits below count only block loads issued
    // after the block they wait for), and round t stages its block t + NB - 1 into the
    // buffer round t - 1 used.  With one key group every split has a block, so its
    // first block is staged without a test (a split shorter than NB - 1 blocks stages
    // its last block again into the spare buffers, which nothing reads).  The compiler
    // still waits for every load before the key-limit reads below.
    const int nmine = kb0 + grp < kb1 ? (kb1 - kb0 - grp + KS - 1) / KS : 0;
#pragma unroll
    for (int j = 0; j < NB - 1; ++j) {
        if constexpr (KS == 1) stage(kb0 + min(j, nmine - 1), j);
        else if (j < nmine) stage(kb0 + grp + j * KS, j);
    }

    // smallest key limit of the wave's 16 rows (lanes 0-15 hold them): blocks below it
    // need no per-key mask.  Read lane by lane into a scalar, so that the per-block
    // test is a scalar branch.
    int lim_w = __builtin_amdgcn_readlane(lim, 0);
#pragma unroll
    for (int i = 1; i < 16; ++i) lim_w = min(lim_w, __builtin_amdgcn_readlane(lim, i));

    float mrun = -INFINITY, lrun = 0.f;
    f32x4_t oacc[ND];
#pragma unroll
    for (int dt = 0; dt < ND; ++dt) oacc[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const int krow0 = 8 * (r >> 2) + (r & 3);   // + 4t: the key this lane reads for tile t

    // every group runs the same number of rounds (the barriers line up); a group
    // whose block lies past the split's range only stages and waits
    const int rounds = (max(kb1 - kb0, 0) + KS - 1) / KS;
    for (int t = 0; t < rounds; ++t) {
        const int kb = kb0 + grp + t * KS;
        const int cur = t % NB;
        // this wave's loads of block t have landed once at most LPW per block staged
        // after it are outstanding (loads complete in issue order, and the loop issues
        // no other vector-memory operations); the barrier then makes every wave's
        // loads visible and frees the buffer round t - 1 read.  No workgroup fence:
        // with loads into LDS in flight it would wait for all of them.
        const int after = min(NB - 2, nmine - 1 - t);
        if (kb < kb1 && kb * 32 + 32 > a.T) {  // the block holding T: the group's last
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            zero_tail(kb, cur);                 // before the barrier, so no other wave reads first
        }
        if (NB > 3 && after >= 2) asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(2 * LPW) : "memory");
        else if (NB > 2 && after >= 1) asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(LPW) : "memory");
        else asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
        if (t + NB - 1 < nmine) stage(kb + (NB - 1) * KS, (t + NB - 1) % NB);
        if (kb >= kb1) continue;
        const char* Kb = lds + (grp * NB + cur) * BUF;
        const char* Vb = Kb + KPLANE;
        const int k0 = kb * 32;

        f32x4_t s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < NC; ++c) {
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                const int key = krow0 + 4 * t;
                const int off = key * (DH * 2) + (((4 * c + g) ^ (swz_k(key) & (KCOLS - 1))) << 4);
                const u32x4_t kf = *(const u32x4_t*)(Kb + off);
                f32x4_t& sa = t ? s1 : s0;
                sa = mfma_f16(kf, qf[c][0], sa);
                sa = mfma_f16(kf, qf[c][1], sa);
            }
        }

        // unscaled scores of keys k0 + 8g + j (j = 0..7); keys past a row's limit -> -inf
        float sv[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            sv[i] = s0[i];
            sv[4 + i] = s1[i];
        }
        if (k0 + 32 > lim_w) {                  // some row of the wave stops inside the block
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int key0 = k0 + 8 * g + i;
                if (key0 >= lim) sv[i] = -INFINITY;
                if (key0 + 4 >= lim) sv[4 + i] = -INFINITY;
            }
        }
        // the row's block maximum over its four lane groups (lanes l, l ^ 16, l ^ 32,
        // l ^ 48): each swap hands a lane its partner's value, and max is symmetric
        float bm = fmaxf(fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3])),
                         fmaxf(fmaxf(sv[4], sv[5]), fmaxf(sv[6], sv[7])));
        {
            const auto w32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(bm), __float_as_uint(bm), false, false);
            bm = fmaxf(__uint_as_float(w32[0]), __uint_as_float(w32[1]));
            const auto w16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(bm), __float_as_uint(bm), false, false);
            bm = fmaxf(__uint_as_float(w16[0]), __uint_as_float(w16[1]));
        }
        const float bms = bm * sl2;             // log2-domain block maximum (sl2 > 0)
        // Lazy rescaling: the reference maximum mrun moves only when some row of the
        // wave exceeds it by more than ATTN_SLACK (and on a row's first unmasked key),
        // so the probabilities stay <= 2^ATTN_SLACK and most blocks skip the rescale.
        // O, l and m are exact for any reference value; the split merge uses the same m.
        if (__builtin_expect(__builtin_amdgcn_ballot_w64(bms > mrun + ATTN_SLACK) != 0, 0)) {
            const float mnew = fmaxf(mrun, bms);
            const float alpha = (mnew == -INFINITY) ? 1.f : __builtin_amdgcn_exp2f(mrun - mnew);
            lrun *= alpha;
#pragma unroll
            for (int dt = 0; dt < ND; ++dt)
#pragma unroll
                for (int i = 0; i < 4; ++i) oacc[dt][i] *= alpha;
            mrun = mnew;
        }
        // a row with no unmasked key yet keeps m = -inf; its masked scores give p = 0
        const float mref = (mrun == -INFINITY) ? 0.f : mrun;
        float ps;
        uint32_t phi[4], plo[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            // v_exp_f32 directly: the arguments are <= ATTN_SLACK (or -inf); results below
            // 2^-126 (flushed to zero) are the only ones that differ from exp2f
            const float p0 = __builtin_amdgcn_exp2f(fmaf(sv[2 * e], sl2, -mref));
            const float p1 = __builtin_amdgcn_exp2f(fmaf(sv[2 * e + 1], sl2, -mref));
            ps = e ? ps + (p0 + p1) : p0 + p1;
            // hi = fp16 toward zero, lo = the remainder toward zero
            const auto h = __builtin_amdgcn_cvt_pkrtz(p0, p1);
            const auto l = __builtin_amdgcn_cvt_pkrtz(p0 - (float)h[0], p1 - (float)h[1]);
            phi[e] = __builtin_bit_cast(uint32_t, h);
            plo[e] = __builtin_bit_cast(uint32_t, l);
        }
        lrun += ps;
        const u32x4_t ph = {phi[0], phi[1], phi[2], phi[3]};
        const u32x4_t pl = {plo[0], plo[1], plo[2], plo[3]};
        // (V^T of keys past T was zeroed when the block holding T was staged)
#pragma unroll
        for (int dt = 0; dt < ND; ++dt) {
            const int dim = 16 * dt + r;
            const u32x4_t vf = *(const u32x4_t*)(Vb + dim * 64 + ((g ^ ((dim >> 2) & 3)) << 4));
            oacc[dt] = mfma_f16(vf, ph, oacc[dt]);
            oacc[dt] = mfma_f16(vf, pl, oacc[dt]);
        }
    }

    float l = lrun;
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);
    if constexpr (KS > 1) {
        // merge the key groups in group order: O = sum_k o_k 2^(m_k - M), L = sum_k l_k 2^(m_k - M)
        __syncthreads();                        // every group is done with its staging buffers
        float* o_sm = (float*)lds;              // [KS][QG * 16][MLD]
        float* m_sm = o_sm + KS * QG * 16 * MLD;
        float* l_sm = m_sm + KS * QG * 16;
        const int rec = grp * QG * 16 + qw * 16 + r;
#pragma unroll
        for (int dt = 0; dt < ND; ++dt)
#pragma unroll
            for (int i = 0; i < 4; ++i) o_sm[rec * MLD + 16 * dt + 4 * g + i] = oacc[dt][i];
        if (g == 0) {
            m_sm[rec] = mrun;
            l_sm[rec] = l;
        }
        __syncthreads();
        const int row0 = z * 16 * QG;
        for (int idx = threadIdx.x; idx < QG * 16 * (DH / 4); idx += blockDim.x) {
            const int q = idx / (DH / 4), d0 = 4 * (idx % (DH / 4));
            float mx = -INFINITY;
#pragma unroll
            for (int k = 0; k < KS; ++k) mx = fmaxf(mx, m_sm[k * QG * 16 + q]);
            float L = 0.f;
            float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
            for (int k = 0; k < KS; ++k) {
                const float mk = m_sm[k * QG * 16 + q];
                const float e = (mk == -INFINITY) ? 0.f : exp2f(mk - mx);
                const float* ok = o_sm + (k * QG * 16 + q) * MLD + d0;
                L += l_sm[k * QG * 16 + q] * e;
                o.x += ok[0] * e; o.y += ok[1] * e; o.z += ok[2] * e; o.w += ok[3] * e;
            }
            if (a.nsplit == 1) {
                const float inv = 1.f / L;
                xfrag_store4<false>(a.o, row0 + q, h * DH + d0, a.KCx,
                                    make_float4(o.x * inv, o.y * inv, o.z * inv, o.w * inv));
            } else {
                float* op = a.opart + (((size_t)split * a.rows_ld + row0 + q) * a.H + h) * DH;
                *(float4*)(op + d0) = o;
                if (d0 == 0) {
                    float* ml = a.mlpart + (((size_t)split * a.rows_ld + row0 + q) * a.H + h) * 2;
                    ml[0] = mx;
                    ml[1] = L;
                }
            }
        }
        return;
    }
    if (a.nsplit == 1) {
        const float inv = 1.f / l;
#pragma unroll
        for (int dt = 0; dt < ND; ++dt)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                xfrag_store<false>(a.o, row, h * DH + 16 * dt + 4 * g + i, a.KCx, oacc[dt][i] * inv);
    } else {
        float* op = a.opart + (((size_t)split * a.rows_ld + row) * a.H + h) * DH;
#pragma unroll
        for (int dt = 0; dt < ND; ++dt)
            *(float4*)(op + 16 * dt + 4 * g) = make_float4(oacc[dt][0], oacc[dt][1], oacc[dt][2], oacc[dt][3]);
        if (g == 0) {
            float* ml = a.mlpart + (((size_t)split * a.rows_ld + row) * a.H + h) * 2;
            ml[0] = mrun;
            ml[1] = l;
        }
    }
}

// Merge key-range splits: O = sum_s o_s 2^(m_s - M) / sum_s l_s 2^(m_s - M).
// 32 lanes per (row, head), four consecutive dims per lane (head dims <= 128);
// ATTN_MERGE_PAIRS (row, head) pairs per workgroup: 4, so that a 32-row window over
// 32 heads gives every CU one workgroup (LLaDA-8B, 32 rows: attention + merge 13.8 ->
// 12.1 us per layer against 8 pairs and 128 workgroups; 2 pairs and 512 workgroups:
// no gain).
constexpr int ATTN_MERGE_PAIRS = 4;
template <bool XF32>
__global__ void __launch_bounds__(32 * ATTN_MERGE_PAIRS) attn_combine_kernel(AttnArgs a, int rows, int DH) {
    constexpr int MAXS = 16;                                   // = the runtime's split cap
    const int pair = blockIdx.x * ATTN_MERGE_PAIRS + (threadIdx.x >> 5);
    const int l = threadIdx.x & 31;
    if (pair >= rows * a.H) return;
    const int h = pair % a.H, row = pair / a.H;
    const size_t stride_s = (size_t)a.rows_ld * a.H;          // (row, head) records per split
    const size_t rec = (size_t)row * a.H + h;
    const int d0 = 4 * l;
    const bool has_d = d0 < DH;
    // every split's (m, l) and output loads go out before any is used: one memory
    // round trip
    float2 ml[MAXS];
    float4 v[MAXS];
#pragma unroll
    for (int s = 0; s < MAXS; ++s) {
        ml[s] = (s < a.nsplit) ? *(const float2*)(a.mlpart + (s * stride_s + rec) * 2)
                               : make_float2(-INFINITY, 0.f);
        v[s] = (s < a.nsplit && has_d) ? *(const float4*)(a.opart + (s * stride_s + rec) * DH + d0)
                                       : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    float mx = -INFINITY;
#pragma unroll
    for (int s = 0; s < MAXS; ++s) mx = fmaxf(mx, ml[s].x);
    float w[MAXS], L = 0.f;
#pragma unroll
    for (int s = 0; s < MAXS; ++s) {
        w[s] = (ml[s].x == -INFINITY) ? 0.f : exp2f(ml[s].x - mx);
        L += ml[s].y * w[s];
    }
    const float inv = 1.f / L;
    if (!has_d) return;
    float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int s = 0; s < MAXS; ++s) {
        o.x += v[s].x * w[s]; o.y += v[s].y * w[s]; o.z += v[s].z * w[s]; o.w += v[s].w * w[s];
    }
    xfrag_store4<XF32>(a.o, row, h * DH + d0, a.KCx, make_float4(o.x * inv, o.y * inv, o.z * inv, o.w * inv));
}

// fp32 path (small models): one wave per (row, head); lanes stride over keys with
// a lane-local online softmax, merged across lanes by a butterfly.
template <int DH>
__global__ void __launch_bounds__(64) attn_f32_kernel(AttnArgs a) {
    const int lane = threadIdx.x;
    const int row = blockIdx.x, h = blockIdx.y;
    const int ld = a.H * DH;
    const float* qp = (const float*)a.q + (size_t)row * ld + h * DH;
    const int hk = h / a.G;                                  // K/V head of this query head
    const float* Kp = (const float*)a.K + (size_t)hk * a.Cs * DH;
    const float* Vp = (const float*)a.Vt + (size_t)hk * DH * a.Cs;
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
