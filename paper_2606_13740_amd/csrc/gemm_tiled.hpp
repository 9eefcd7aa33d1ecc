// Tiled GEMM for many token rows (prompt processing): Y = X W^T with bf16 or int8
// weights, where the streaming kernel's waves each fetch their own operand fragments
// and the matrix cores stay ~30% busy.
//
// Workgroup = 8 waves = 2 row halves x 4 token quarters; it owns 16 row tiles x TT
// token tiles (bf16: 256 rows x 256 tokens; int8: 256 x 128) and a K range (split-K
// over grid.y, for the residual projections' partial sums).  Each K step (one weight
// chunk: 32 columns bf16, 64 int8) its 16 weight chunks and the token tiles'
// activation chunks (hi, lo planes; two per token tile for int8) are copied once into
// LDS with direct global->LDS loads, three stages deep, and every wave multiplies its
// 8 row tiles by its token tiles from there: 64 MFMAs per 16 KiB of LDS reads, against
// 16 KiB of L1/L2 fetches per 64 MFMAs in the streaming layouts.  The packed formats
// are the streaming kernel's (chunks are already in MFMA fragment order, so an LDS
// chunk is read with one 16-byte load per lane; int8 is widened to bf16 after the
// read).  Results go through the same epilogues, in four passes of TT / 4 token tiles.
#pragma once

#include "gemm.hpp"

namespace dllm {

typedef __attribute__((address_space(3))) void lds_void;

template <int WT>
struct TiledShape {
    static_assert(WT == WT_BF16 || WT == WT_I8, "tiled GEMM: bf16 or int8 weights");
    static constexpr int XPER = WTraits<WT>::XPER;   // activation chunks per weight chunk
    static constexpr int RT = 16;                    // row tiles per workgroup
    static constexpr int WM = 4 / XPER;              // token tiles per wave
    static constexpr int TT = 4 * WM;                // token tiles per workgroup
    static constexpr int WR = 8;                     // row tiles per wave
    static constexpr int S = 3;                      // LDS stages
    static constexpr int WB = RT * 1024;             // weight bytes per stage
    static constexpr int XB = TT * XPER * 2048;      // activation bytes per stage (hi + lo)
    static constexpr int SB = WB + XB;
    static constexpr int LOADS = (RT + 2 * XPER * TT) / 8;   // 1 KiB global->LDS loads per wave and stage
    static constexpr int LDY = 16 * WM + 1;
};

// m_tiles: token tiles of X (its rows / 16, a multiple of 4); rows past them are
// never read (loads clamp to the last tile) and never written.
template <int WT, class Epi>
__global__ void __launch_bounds__(512) gemm_tiled_kernel(GemmArgs g, Epi epi, int m_tiles) {
    using T = TiledShape<WT>;
    constexpr int XPER = T::XPER;
    static_assert(T::LOADS * 8 == T::RT + 2 * XPER * T::TT, "stage loads must split evenly over the waves");
    static_assert(16 * T::RT * T::LDY * 4 <= T::S * T::SB, "epilogue tile must fit the stage buffers");
    __shared__ __attribute__((aligned(1024))) char sm[T::S * T::SB];
    constexpr int ESM = Epi::kSmem > 0 ? Epi::kSmem : 16;
    __shared__ __align__(16) char esm[ESM];

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wr = wave & 1, wq = wave >> 1;
    const int nt0 = blockIdx.x * T::RT, mt0 = blockIdx.z * T::TT;
    const int KC = g.KCw;
    const unsigned KS = gridDim.y;
    const int c0 = (int)((blockIdx.y * (unsigned)KC) / KS), c1 = (int)(((blockIdx.y + 1) * (unsigned)KC) / KS);

    // stage slot i: i < RT the weight chunk of row tile nt0 + i, else activation chunk
    // q = i - RT: token tile q / (2 XPER), column half (q / 2) % XPER, plane q % 2;
    // wave w copies slots w + 8j
    auto stage = [&](int c, int buf) {
        char* base = sm + buf * T::SB;
#pragma unroll
        for (int j = 0; j < T::LOADS; ++j) {
            const int i = wave + 8 * j;
            const char* src;
            char* dst;
            if (j < T::RT / 8) {
                const int nt = min(nt0 + i, g.n_tiles - 1);
                src = (const char*)g.W + (((size_t)nt * KC + c) * 64 + lane) * 16;
                dst = base + i * 1024;
            } else {
                const int q = i - T::RT, tt = q / (2 * XPER), h = (q >> 1) % XPER, pl = q & 1;
                const int mt = min(mt0 + tt, m_tiles - 1);
                src = (const char*)g.X + ((size_t)mt * g.KCx + c * XPER + h) * 2048 + pl * 1024 + lane * 16;
                dst = base + T::WB + q * 1024;
            }
            __builtin_amdgcn_global_load_lds((const void*)src, (lds_void*)dst, 16, 0, 0);
        }
    };

    f32x4_t acc[T::WR][T::WM];
#pragma unroll
    for (int f = 0; f < T::WR; ++f)
#pragma unroll
        for (int t = 0; t < T::WM; ++t) acc[f][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    if (c1 > c0) {
        // every step issues one stage (past the end: the last chunk again, into a
        // buffer nobody reads), so each wave always has exactly LOADS loads of the
        // following stage in flight when it waits for the current one
        stage(c0, 0);
        stage(min(c0 + 1, c1 - 1), 1);
        for (int c = c0; c < c1; ++c) {
            const int cur = (c - c0) % T::S;
            // this wave's copies of stage c have landed (the next stage's may not) and
            // its LDS reads are done; after the barrier every wave's copies have landed
            // and nobody reads the buffer refilled next.  (__syncthreads would also wait
            // for the next stage's copies: the fence before its barrier waits for all
            // outstanding vector memory operations.)
            asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(T::LOADS) : "memory");
            stage(min(c + 2, c1 - 1), (c - c0 + 2) % T::S);
            const char* Wb = sm + cur * T::SB;
            const char* Xb = Wb + T::WB;
            u32x4_t xh[T::WM][XPER], xl[T::WM][XPER];
#pragma unroll
            for (int t = 0; t < T::WM; ++t)
#pragma unroll
                for (int h = 0; h < XPER; ++h) {
                    const char* xp = Xb + (((T::WM * wq + t) * XPER + h) * 2) * 1024 + lane * 16;
                    xh[t][h] = *(const u32x4_t*)xp;
                    xl[t][h] = *(const u32x4_t*)(xp + 1024);
                }
#pragma unroll
            for (int f = 0; f < T::WR; ++f) {
                const u32x4_t raw = *(const u32x4_t*)(Wb + (T::WR * wr + f) * 1024 + lane * 16);
                u32x4_t w[XPER];
                if constexpr (WT == WT_I8) {
                    w[0] = i8x8_to_bf16x8(raw[0], raw[1]);
                    w[XPER - 1] = i8x8_to_bf16x8(raw[2], raw[3]);
                } else {
                    w[0] = raw;
                }
#pragma unroll
                for (int h = 0; h < XPER; ++h)
#pragma unroll
                    for (int t = 0; t < T::WM; ++t) {
                        acc[f][t] = mfma_bf16(w[h], xh[t][h], acc[f][t]);
                        acc[f][t] = mfma_bf16(w[h], xl[t][h], acc[f][t]);
                    }
            }
        }
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    }
    __syncthreads();

    // epilogue: four passes of WM token tiles over the stage buffers (rows 0..255 of Y)
    float* Y = (float*)sm;
    const int nrows = 16 * max(0, min(T::RT, g.n_tiles - nt0));
    const int r = lane & 15, gq = lane >> 4;
    for (int p = 0; p < T::TT / T::WM; ++p) {
        const int mtp = mt0 + T::WM * p;
        if (mtp >= m_tiles || nrows == 0) break;
        const int mcols = 16 * min(T::WM, m_tiles - mtp);
        if (wq == p) {
#pragma unroll
            for (int f = 0; f < T::WR; ++f)
#pragma unroll
                for (int t = 0; t < T::WM; ++t)
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        Y[(16 * (T::WR * wr + f) + 4 * gq + i) * T::LDY + 16 * t + r] = acc[f][t][i];
        }
        __syncthreads();
        if (g.wscale != nullptr || g.bias != nullptr) {
            for (int idx = threadIdx.x; idx < nrows * mcols; idx += blockDim.x) {
                const int n = idx / mcols, m = idx % mcols;
                float y = Y[n * T::LDY + m];
                if (g.wscale != nullptr) y *= g.wscale[nt0 * 16 + n];
                if (g.bias != nullptr) y += g.bias[nt0 * 16 + n];
                Y[n * T::LDY + m] = y;
            }
            __syncthreads();
        }
        typename Epi::Pre pre;
        epi.fetch(pre, nt0 * 16, nrows, mtp * 16, mcols);
        epi.stage(pre, esm, nt0 * 16, nrows, mtp * 16, mcols);
        __syncthreads();
        epi(Y, T::LDY, nt0 * 16, nrows, mtp * 16, mcols, blockIdx.x, esm, NoScale{});
        __syncthreads();
    }
}

// Split-K finish of the tiled kernel for the QKV projection of short prompts (whose
// 256 x 256 tiles alone leave the chip half idle): each workgroup sums the KS partial
// slices P[s][m][n] of a 256-row x 64-token block in slice order into an LDS tile,
// adds the bias once, and runs the projection's epilogue on it, as the tiled kernel
// does with its own sums.
template <class Epi>
__global__ void __launch_bounds__(256) split_epilogue_kernel(const float* P, int ks, int rows, int ldn, int n_tiles,
                                                             int m_tiles, const float* bias, Epi epi) {
    constexpr int RT = 16, WM = 4, LDY = 16 * WM + 1;
    __shared__ float Y[16 * RT * LDY];
    constexpr int ESM = Epi::kSmem > 0 ? Epi::kSmem : 16;
    __shared__ __align__(16) char esm[ESM];
    const int nt0 = blockIdx.x * RT, mt0 = blockIdx.y * WM;
    const int nrows = 16 * min(RT, n_tiles - nt0), mcols = 16 * min(WM, m_tiles - mt0);
    const int n0 = nt0 * 16, m0 = mt0 * 16;
    const size_t slice = (size_t)rows * ldn;
    // four consecutive outputs of one token per thread (16-byte loads along P's rows)
    const int nq = nrows >> 2;
    for (int idx = threadIdx.x; idx < nq * mcols; idx += blockDim.x) {
        const int qd = idx % nq, ml = idx / nq, nl = 4 * qd;
        const float* p = P + (size_t)(m0 + ml) * ldn + n0 + nl;
        float4 v = *(const float4*)p;
        for (int k = 1; k < ks; ++k) {
            const float4 u = *(const float4*)(p + k * slice);
            v.x += u.x; v.y += u.y; v.z += u.z; v.w += u.w;
        }
        if (bias != nullptr) {
            v.x += bias[n0 + nl]; v.y += bias[n0 + nl + 1]; v.z += bias[n0 + nl + 2]; v.w += bias[n0 + nl + 3];
        }
        Y[nl * LDY + ml] = v.x;
        Y[(nl + 1) * LDY + ml] = v.y;
        Y[(nl + 2) * LDY + ml] = v.z;
        Y[(nl + 3) * LDY + ml] = v.w;
    }
    typename Epi::Pre pre;
    epi.fetch(pre, n0, nrows, m0, mcols);
    epi.stage(pre, esm, n0, nrows, m0, mcols);
    __syncthreads();
    epi(Y, LDY, n0, nrows, m0, mcols, blockIdx.x, esm, NoScale{});
}

}  // namespace dllm
