// Small kernels around the GEMMs: embedding gather, LM-head merge, commit,
// weight prepacking / int8 quantisation and the RoPE table.
#pragma once

#include "common.hpp"
#include "gemm.hpp"

namespace dllm {

// ---------------------------------------------------------------------------
// Row-wise RMSNorm operand: given the finished residual row x[m][0..d), write
// the next GEMM's A operand h = x * rsqrt(mean(x^2) + eps) * g into the
// activation fragments.  Each thread holds VPT column groups of 4 values.
// ---------------------------------------------------------------------------
template <int NT>
__device__ __forceinline__ float block_sum(float v, float* red /* NT/64 */) {
    v = warp_sum(v);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < NT / 64; ++w) s += red[w];
    __syncthreads();
    return s;
}

// With ssq != nullptr (RMSNorm folded into the consumer GEMM) the operand is x * g,
// not normalised, and the row's sum of x^2 goes to *ssq for the consumer.  The
// caller loads the gain gv with the row (one memory round trip, not a second one
// after the block sum's barriers).
template <bool XF32, int NT, int VPT>
__device__ __forceinline__ void write_norm_operand(const float4 (&xv)[VPT], const float4 (&gv)[VPT], int m, int d,
                                                   float eps, void* xg, int KCx, float* red, float* ssq = nullptr) {
    float sq = 0.f;
#pragma unroll
    for (int j = 0; j < VPT; ++j) {
        const int n = 4 * (threadIdx.x + j * NT);
        if (n < d) sq += xv[j].x * xv[j].x + xv[j].y * xv[j].y + xv[j].z * xv[j].z + xv[j].w * xv[j].w;
    }
    const float tot = block_sum<NT>(sq, red);
    if (ssq != nullptr && threadIdx.x == 0) *ssq = tot;
    const float rs = ssq != nullptr ? 1.0f : 1.0f / sqrtf(tot / d + eps);
#pragma unroll
    for (int j = 0; j < VPT; ++j) {
        const int n = 4 * (threadIdx.x + j * NT);
        if (n >= d) continue;
        const float4 gg = gv[j];
        xfrag_store4<XF32>(xg, m, n, KCx,
                           make_float4(xv[j].x * rs * gg.x, xv[j].y * rs * gg.y, xv[j].z * rs * gg.z,
                                       xv[j].w * rs * gg.w));
    }
}

// Rows of the residual kernels: NT threads x VPT float4 groups cover d <= 4*NT*VPT.
constexpr int ROW_NT = 1024;
constexpr int ROW_VPT = 2;      // d up to 8192

// Row selection of the LM head (selective logits skipping): row m of M is kept if
// it is flagged (need[m] != 0; every row when need is NULL) and fewer than n_sel
// flagged rows precede it; a kept row's slot is that count.  Returns -1 for a row
// that is not kept.  Every thread of the block gets the same answer.
template <int NT>
__device__ __forceinline__ int lm_slot(const uint8_t* need, int n_sel, int M, int m, float* red) {
    if (need == nullptr) return (m < M && m < n_sel) ? m : -1;
    float c = 0.f;
    for (int i = threadIdx.x; i < m && i < M; i += NT) c += need[i] ? 1.f : 0.f;
    const int before = (int)block_sum<NT>(c, red);
    return (m < M && need[m] && before < n_sel) ? before : -1;
}

// Embedding gather: x[m] = E[id_m] (the MASK id where the mask flag is set) and
// the first layer's normalised operand (or, with ssq, the operand x * g and the
// row's sum of x^2 for an RMSNorm folded into the QKV GEMM).  Padding rows get zeros.
// With slot != nullptr it also records the row's LM-head slot (lm_slot over need /
// n_sel) for the last residual projection, which writes the final operand there.
template <typename ET, bool XF32>
__global__ void __launch_bounds__(ROW_NT)
embed_kernel(const ET* E, const int* tok, const uint8_t* mask, int M, int d, int V, int mask_id, float eps,
             const float* g, float* x, void* xg, int KCx, float* ssq, int ssq_ld, int* slot, const uint8_t* need,
             int n_sel) {
    __shared__ float red[ROW_NT / 64];
    const int m = blockIdx.x;
    if (slot != nullptr) {
        const int sl = lm_slot<ROW_NT>(need, n_sel, M, m, red);
        if (threadIdx.x == 0) slot[m] = sl;
    }
    float4 xv[ROW_VPT], gv[ROW_VPT];
    int id = -1;
    if (m < M) {
        id = (mask != nullptr && mask[m]) ? mask_id : tok[m];
        if (id < 0 || id >= V) id = mask_id;
    }
#pragma unroll
    for (int j = 0; j < ROW_VPT; ++j) {
        const int n = 4 * (threadIdx.x + j * ROW_NT);
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f), gg = v;
        if (n < d) {
            gg = *(const float4*)(g + n);
            if (id >= 0) {
                const ET* row = E + (size_t)id * d + n;
                v = make_float4(to_f32<ET>(row[0]), to_f32<ET>(row[1]), to_f32<ET>(row[2]), to_f32<ET>(row[3]));
            }
            *(float4*)(x + (size_t)m * d + n) = v;
        }
        xv[j] = v;
        gv[j] = gg;
    }
    write_norm_operand<XF32, ROW_NT, ROW_VPT>(xv, gv, m, d, eps, xg, KCx, red,
                                              ssq != nullptr ? ssq + (size_t)m * ssq_ld : nullptr);
}

// Split-K reduction of a residual projection (O or down), one workgroup per row:
//   x[m][n] += sum_ks P[ks][m][n]   (fixed order),
// then the next RMSNorm's normalised operand.  Padding rows get zeros.  With
// `sel` set (the last layer feeding a selective LM head) the operand of a kept row
// goes to its slot (lm_slot) and other rows write none.  KS (the K slices) is a
// template argument so that the slices, the residual and the gain are loaded
// without a condition each, in one round (a select per slice made the compiler
// wait for the first loads before issuing the rest).
template <bool XF32, int KS>
__global__ void __launch_bounds__(ROW_NT)
residual_reduce_kernel(const float* P, int prow, int d, int M, float eps, float* x, const float* g,
                       void* xg, int KCx, bool sel, const uint8_t* need, int n_sel) {
    __shared__ float red[ROW_NT / 64];
    const int m = blockIdx.x;
    float4 xv[ROW_VPT], gv[ROW_VPT];
#pragma unroll
    for (int j = 0; j < ROW_VPT; ++j) {
        const int n = 4 * (threadIdx.x + j * ROW_NT);
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f), gg = v;
        if (n < d && m < M) {
            float4* xp = (float4*)(x + (size_t)m * d + n);
            float4 p[KS];
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) p[ks] = *(const float4*)(P + ((size_t)ks * prow + m) * d + n);
            v = *xp;
            gg = *(const float4*)(g + n);
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                v.x += p[ks].x; v.y += p[ks].y; v.z += p[ks].z; v.w += p[ks].w;
            }
            *xp = v;
        }
        xv[j] = v;
        gv[j] = gg;
    }
    const int dst = sel ? lm_slot<ROW_NT>(need, n_sel, M, m, red) : m;
    if (dst >= 0) write_norm_operand<XF32, ROW_NT, ROW_VPT>(xv, gv, dst, d, eps, xg, KCx, red);
}

// Zeroes the padding columns [kreal, KCx * columns per chunk) of an activation
// fragment buffer for `tiles` token tiles.  No kernel writes those columns and the
// GEMMs multiply them by zero weight columns, so they must hold finite values (zeros):
// a freshly zeroed workspace does, a reused scratch buffer needs this.  One thread per
// 16-byte lane slot of the chunks that hold padding (bf16 hi/lo: 2 planes).
template <bool XF32>
__global__ void __launch_bounds__(256) zero_frag_pad_kernel(void* buf, int tiles, int KCx, int kreal) {
    constexpr int KCOL = XF32 ? 16 : 32;                  // columns per activation chunk
    const int kc0 = kreal / KCOL;                          // first chunk holding padding
    const int nch = KCx - kc0;
    const int planes = XF32 ? 1 : 2;
    const long u = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (nch <= 0 || u >= (long)tiles * nch * 64 * planes) return;
    const int lane = (int)(u % 64);
    const int pl = (int)((u / 64) % planes);
    const int c = (int)((u / (64 * planes)) % nch);
    const int t = (int)(u / (64 * planes * nch));
    const int kc = kc0 + c, g = lane >> 4;
    char* p = (char*)buf + (size_t)(t * KCx + kc) * (XF32 ? 1024 : 2048) + pl * 1024 + lane * 16;
    if (XF32) {
#pragma unroll
        for (int s = 0; s < 4; ++s)
            if (kc * 16 + 4 * s + g >= kreal) ((float*)p)[s] = 0.f;
    } else {
#pragma unroll
        for (int e = 0; e < 8; ++e)
            if (kc * 32 + 8 * g + e >= kreal) ((uint16_t*)p)[e] = 0;
    }
}

// Streaming read of n 16-byte units (measurement helper): grid-stride, 4 loads in flight per lane.
__global__ void __launch_bounds__(256) read_stream_kernel(const u32x4_t* p, size_t n, uint32_t* sink) {
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    uint32_t acc = 0;
    for (; i + 3 * stride < n; i += 4 * stride) {
        const u32x4_t a = ldg16_nt(p + i), b = ldg16_nt(p + i + stride);
        const u32x4_t c = ldg16_nt(p + i + 2 * stride), d = ldg16_nt(p + i + 3 * stride);
        acc ^= a[0] ^ a[1] ^ a[2] ^ a[3] ^ b[0] ^ b[1] ^ b[2] ^ b[3] ^ c[0] ^ c[1] ^ c[2] ^ c[3] ^ d[0] ^ d[1] ^
               d[2] ^ d[3];
    }
    for (; i < n; i += stride) {
        const u32x4_t a = ldg16_nt(p + i);
        acc ^= a[0] ^ a[1] ^ a[2] ^ a[3];
    }
    if (acc == 0x9E3779B9u) *sink = acc;
}

// ---------------------------------------------------------------------------
// LM-head merge across vocabulary tiles -> id, confidence = 1 / sum exp(l - max)
// ---------------------------------------------------------------------------
__device__ __forceinline__ LmPartial lm_merge(LmPartial a, LmPartial b) {
    if (b.arg < 0) return a;
    if (a.arg < 0) return b;
    LmPartial o;
    o.mx = fmaxf(a.mx, b.mx);
    if (a.mx > b.mx) o.arg = a.arg;
    else if (b.mx > a.mx) o.arg = b.arg;
    else o.arg = min(a.arg, b.arg);
    o.s = a.s * expf(a.mx - o.mx) + b.s * expf(b.mx - o.mx);
    o.pad = 0.f;
    return o;
}

// One workgroup per window row m.  With `sel`, row m reads the partials of its LM
// slot (lm_slot); a row without one reports id -1 and confidence 0.
__global__ void __launch_bounds__(64)
lm_combine_kernel(const LmPartial* part, int n_wg, int part_ld, int* out_id, float* out_conf, bool sel,
                  const uint8_t* need, int n_sel, int M) {
    __shared__ float red[1];
    const int lane = threadIdx.x;
    int m = blockIdx.x;
    if (sel) {
        const int slot = lm_slot<64>(need, n_sel, M, blockIdx.x, red);
        if (slot < 0) {
            if (lane == 0) {
                if (out_id) out_id[blockIdx.x] = -1;
                if (out_conf) out_conf[blockIdx.x] = 0.f;
            }
            return;
        }
        m = slot;
    }
    // Lane l merges records l, l + 64, l + 128, ... in that order.  The loads of a round
    // go out together, unconditionally (an index past the last record reloads the last
    // one, which the merge then skips): with a select per load the compiler waited for
    // the first loads before issuing the rest.
    LmPartial acc{-INFINITY, -1, 0.f, 0.f};
    constexpr int R = 16;
    for (int w0 = lane; w0 < n_wg; w0 += 64 * R) {
        LmPartial q[R];
#pragma unroll
        for (int j = 0; j < R; ++j) q[j] = part[(size_t)min(w0 + 64 * j, n_wg - 1) * part_ld + m];
#pragma unroll
        for (int j = 0; j < R; ++j)
            if (w0 + 64 * j < n_wg) acc = lm_merge(acc, q[j]);
    }
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        LmPartial o;
        o.mx = __shfl_xor(acc.mx, off);
        o.arg = __shfl_xor(acc.arg, off);
        o.s = __shfl_xor(acc.s, off);
        o.pad = 0.f;
        // combine in lane order so every lane computes the same merge
        acc = (lane & off) ? lm_merge(o, acc) : lm_merge(acc, o);
    }
    if (lane == 0) {
        if (out_id) out_id[blockIdx.x] = acc.arg;
        if (out_conf) out_conf[blockIdx.x] = 1.0f / acc.s;
    }
}

// ---------------------------------------------------------------------------
// Commit: top-k masked positions of a segment by confidence (ties -> lower
// position).  Every thread ranks its positions against the whole segment.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256)
commit_kernel(const float* conf, const int* id, int* tok, uint8_t* mask, int seg_begin, int seg_len,
              int k, int* committed, int* n_committed) {
    __shared__ float c_s[1024];
    __shared__ uint8_t m_s[1024];
    __shared__ int cnt;
    if (threadIdx.x == 0) cnt = 0;
    __syncthreads();
    int local = 0;
    for (int i = threadIdx.x; i < seg_len; i += blockDim.x) {
        const uint8_t mk = mask[seg_begin + i];
        m_s[i] = mk;
        c_s[i] = conf[seg_begin + i];
        local += mk ? 1 : 0;
    }
    atomicAdd(&cnt, local);
    __syncthreads();
    for (int i = threadIdx.x; i < seg_len; i += blockDim.x) {
        if (!m_s[i]) continue;
        const float ci = c_s[i];
        int rank = 0;
        for (int j = 0; j < seg_len; ++j)
            if (m_s[j] && (c_s[j] > ci || (c_s[j] == ci && j < i))) ++rank;
        if (rank < k) {
            const int p = seg_begin + i;
            tok[p] = id[p];
            mask[p] = 0;
            if (committed) committed[rank] = p;
        }
    }
    if (threadIdx.x == 0 && n_committed) *n_committed = min(k, cnt);
}

// ---------------------------------------------------------------------------
// Staged token stabilisation over one segment (one thread per position, <= 1024):
// state 0 invisible (masked), 1 visible, 2 stable.  Invisible positions at or
// above tv become visible (taking their predicted id); if there is none, the
// most confident invisible position does (ties: lower position); a visible
// position becomes stable when this step predicts the id it holds with a
// confidence at or above ts (stability is a property of the held token).  The
// promoted positions are written in ascending order.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(1024)
commit_staged_kernel(const float* conf, const int* id, int* tok, uint8_t* mask, uint8_t* state, int seg_begin,
                     int seg_len, float tv, float ts, int* promoted, int* n_promoted) {
    __shared__ unsigned long long best;
    __shared__ int wsum[16];
    const int i = threadIdx.x;
    const bool in = i < seg_len;
    const int p = seg_begin + i;
    const uint8_t st = in ? state[p] : (uint8_t)2;
    const float c = in ? conf[p] : 0.f;
    const int pid = in ? id[p] : 0;
    const int held = in ? tok[p] : 0;
    const bool cand = in && st == 0;
    if (i == 0) best = 0ull;
    const bool vis = cand && c >= tv;
    const int nvis = __syncthreads_count(vis);     // also orders the reset of `best`
    bool prom = vis;
    if (nvis == 0) {
        // confidences are >= 0, so their bit patterns order like the values; the low
        // word (>= 1) prefers the lower position and marks that a candidate exists
        if (cand) atomicMax(&best, ((unsigned long long)__float_as_uint(c) << 32) | (unsigned)(1024 - i));
        __syncthreads();
        prom = cand && best != 0ull && (int)(1024u - (unsigned)(best & 0xFFFFFFFFull)) == i;
    }
    uint8_t ns = prom ? (uint8_t)1 : st;
    if (ns == 1 && c >= ts && (prom || pid == held)) ns = 2;
    if (in) {
        if (prom) {
            tok[p] = pid;
            mask[p] = 0;
        }
        if (ns != st) state[p] = ns;
    }
    const unsigned long long bal = __ballot(prom);
    const int lane = i & 63, w = i >> 6;
    if (lane == 0) wsum[w] = __popcll(bal);
    __syncthreads();
    int off = 0;
    for (int j = 0; j < w; ++j) off += wsum[j];
    if (prom && promoted != nullptr) promoted[off + __popcll(bal & ((1ull << lane) - 1ull))] = p;
    if (i == 0 && n_promoted != nullptr) {
        int t = 0;
        for (int j = 0; j < (int)(blockDim.x >> 6); ++j) t += wsum[j];
        *n_promoted = t;
    }
}

// ---------------------------------------------------------------------------
// Weight prepacking into MFMA chunks.  Packed row r takes source row
// rowmap(r) of one of up to three source matrices (or zeros for padding).
// ---------------------------------------------------------------------------
enum RowMap : int { MAP_IDENT = 0, MAP_QKV = 1, MAP_GATEUP = 2 };

struct PackSrc {
    const void* src[3];
    int kind;
    int N;        // real packed rows
    int K;        // real columns
    int d, Dh;    // for MAP_QKV: Q rows (H * Dh) and head size
    int dkv;      // for MAP_QKV: K and V rows each (Hkv * Dh)
};

// MAP_QKV packed rows: [Q: d rows | K: dkv rows | V: dkv rows]; inside every Q or K
// head, packed row 2i is dim i and 2i+1 is dim i + Dh/2 (a RoPE pair is adjacent).
__device__ __forceinline__ const void* src_row(const PackSrc& p, int r, int& row) {
    if (r >= p.N) return nullptr;
    if (p.kind == MAP_IDENT) { row = r; return p.src[0]; }
    if (p.kind == MAP_GATEUP) { row = r >> 1; return p.src[r & 1]; }
    const int seg = r < p.d ? 0 : (r < p.d + p.dkv ? 1 : 2);
    const int rr = r - (seg == 0 ? 0 : (seg == 1 ? p.d : p.d + p.dkv));
    if (seg == 2) { row = rr; return p.src[2]; }
    const int h = rr / p.Dh, w = rr - h * p.Dh;
    row = h * p.Dh + (w >> 1) + (w & 1) * (p.Dh >> 1);   // adjacent packed rows = RoPE pair
    return p.src[seg];
}

// Q/K/V biases (fp32 vectors in p.src[0..2]) in packed-row order; padding rows 0.
__global__ void __launch_bounds__(256) pack_bias_kernel(PackSrc p, int n_rows_padded, float* out) {
    const int r = blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= n_rows_padded) return;
    int row = 0;
    const float* src = (const float*)src_row(p, r, row);
    out[r] = src ? src[row] : 0.f;
}

// int8 quantiser (per output row, decided in fp32): s = max|w| / 127 and
// q = round-half-even(w / s) clamped to [-127, 127], both divisions correctly
// rounded; a zero row has s = 0 and all codes 0.
__device__ __forceinline__ float i8_scale(float amax) { return __fdiv_rn(amax, 127.0f); }
__device__ __forceinline__ int i8_code(float x, float s) {
    if (!(s > 0.f)) return 0;
    const int q = (int)rintf(__fdiv_rn(x, s));
    return max(-127, min(127, q));
}

// One thread per 16-byte lane slot.  ST: source element type (float / uint16_t bf16).
template <int WT, typename ST>
__global__ void __launch_bounds__(256)
pack_kernel(PackSrc p, int n_tiles, int KCw, u32x4_t* out, const float* scale) {
    const size_t u = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const size_t total = (size_t)n_tiles * KCw * 64;
    if (u >= total) return;
    const int lane = (int)(u & 63);
    const size_t ch = u >> 6;
    const int kc = (int)(ch % KCw);
    const int nt = (int)(ch / KCw);
    const int r = nt * 16 + (lane & 15), g = lane >> 4;
    int row = 0;
    const ST* src = (const ST*)src_row(p, r, row);
    u32x4_t v = {0u, 0u, 0u, 0u};
    if (src != nullptr) {
        const ST* s = src + (size_t)row * p.K;
        if constexpr (WT == WT_BF16) {
            uint16_t e[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int k = kc * 32 + 8 * g + i;
                e[i] = (k < p.K) ? f32_to_bf16(to_f32<ST>(s[k])) : (uint16_t)0;
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] = (uint32_t)e[2 * i] | ((uint32_t)e[2 * i + 1] << 16);
        } else if constexpr (WT == WT_F32) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int k = kc * 16 + 4 * q + g;
                v[q] = __float_as_uint((k < p.K) ? to_f32<ST>(s[k]) : 0.f);
            }
        } else {
            const float sc = scale[r];
            uint32_t b[16];
#pragma unroll
            for (int hh = 0; hh < 2; ++hh)
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int k = kc * 64 + 32 * hh + 8 * g + e;
                    const int qv = (k < p.K) ? i8_code(to_f32<ST>(s[k]), sc) : 0;
                    b[8 * hh + e] = (uint32_t)(qv & 0xFF);
                }
#pragma unroll
            for (int i = 0; i < 4; ++i)
                v[i] = b[4 * i] | (b[4 * i + 1] << 8) | (b[4 * i + 2] << 16) | (b[4 * i + 3] << 24);
        }
    }
    out[u] = v;
}

// Q4_0 prepack: one thread per lane slot of a 512-byte chunk (16 rows x 64
// columns = two 32-column blocks): the lane's 8 codes of each block in the dword
// order q4_unpack reads, and (lanes of lane group 0) the two fp16 scales of its row
// at qs[((nt * KCw + kc) * 16 + row) * 2 + block].
template <typename ST>
__global__ void __launch_bounds__(256)
pack_q4_kernel(PackSrc p, int n_tiles, int KCw, u32x2_t* out, uint16_t* qs) {
    const size_t u = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const size_t total = (size_t)n_tiles * KCw * 64;
    if (u >= total) return;
    const int lane = (int)(u & 63);
    const size_t ch = u >> 6;
    const int kc = (int)(ch % KCw);
    const int nt = (int)(ch / KCw);
    const int r = nt * 16 + (lane & 15), g = lane >> 4;
    int row = 0;
    const ST* src = (const ST*)src_row(p, r, row);
    u32x2_t v = {0x88888888u, 0x88888888u};     // padding rows: code 8 = weight 0
    uint16_t sc[2] = {0, 0};
    if (src != nullptr) {
        const ST* s = src + (size_t)row * p.K;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int k0 = kc * 64 + 32 * h;
            float d, inv;
            q4_block<ST>(s, k0, p.K, d, inv);
            uint32_t w = 0;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int k = k0 + 8 * g + e;
                const float x = (k < p.K) ? to_f32<ST>(s[k]) : 0.f;
                w |= q4_code(x, inv) << ((e & 1) ? 16 + 4 * (e >> 1) : 4 * (e >> 1));
            }
            v[h] = w;
            sc[h] = f32_to_f16_bits(d);
        }
    }
    out[u] = v;
    if (g == 0) *(uint32_t*)(qs + ((size_t)(nt * KCw + kc) * 16 + (lane & 15)) * 2) = sc[0] | ((uint32_t)sc[1] << 16);
}

// Q4_0 quantisation to plain row-major arrays (the converter's output, and the
// form the quantiser is checked in): one thread per (row, 32-column block);
// codes [rows][nb * 32] one byte each (padding columns quantised as 0), scales
// [rows][nb] fp16 bits.
template <typename ST>
__global__ void __launch_bounds__(256)
quantize_q4_kernel(const ST* w, int rows, int K, uint8_t* codes, uint16_t* scales) {
    const int nb = (K + 31) / 32;
    const long t = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (long)rows * nb) return;
    const int r = (int)(t / nb), b = (int)(t % nb);
    const ST* s = w + (size_t)r * K;
    float d, inv;
    q4_block<ST>(s, 32 * b, K, d, inv);
    for (int e = 0; e < 32; ++e) {
        const int k = 32 * b + e;
        codes[(size_t)r * nb * 32 + k] = (uint8_t)q4_code((k < K) ? to_f32<ST>(s[k]) : 0.f, inv);
    }
    scales[(size_t)r * nb + b] = f32_to_f16_bits(d);
}

// Per packed row: s = max |w| / 127 (fp32, correctly rounded division).
template <typename ST>
__global__ void __launch_bounds__(256) row_scale_kernel(PackSrc p, int n_rows_padded, float* scale) {
    __shared__ float red[4];
    const int r = blockIdx.x;
    int row = 0;
    const ST* src = (const ST*)src_row(p, r, row);
    float mx = 0.f;
    if (src != nullptr) {
        const ST* s = src + (size_t)row * p.K;
        for (int k = threadIdx.x; k < p.K; k += blockDim.x) mx = fmaxf(mx, fabsf(to_f32<ST>(s[k])));
    }
    mx = warp_max(mx);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = mx;
    __syncthreads();
    if (threadIdx.x == 0 && r < n_rows_padded)
        scale[r] = i8_scale(fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3])));
}

// int8 quantisation to plain row-major arrays (the converter's output, and the form
// the quantiser is checked in): one workgroup per row; codes [rows][K], scales [rows].
template <typename ST>
__global__ void __launch_bounds__(256)
quantize_i8_kernel(const ST* w, int K, int8_t* codes, float* scales) {
    __shared__ float red[4];
    __shared__ float s_sh;
    const int r = blockIdx.x;
    const ST* row = w + (size_t)r * K;
    float mx = 0.f;
    for (int k = threadIdx.x; k < K; k += blockDim.x) mx = fmaxf(mx, fabsf(to_f32<ST>(row[k])));
    mx = warp_max(mx);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = mx;
    __syncthreads();
    if (threadIdx.x == 0) {
        s_sh = i8_scale(fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3])));
        scales[r] = s_sh;
    }
    __syncthreads();
    const float sc = s_sh;
    for (int k = threadIdx.x; k < K; k += blockDim.x) codes[(size_t)r * K + k] = (int8_t)i8_code(to_f32<ST>(row[k]), sc);
}

// (cos, sin) of pos * base^(-2j/Dh), evaluated in double.
__global__ void __launch_bounds__(256) rope_table_kernel(float2* t, int max_pos, int half, double base) {
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (size_t)max_pos * half) return;
    const int j = (int)(i % half);
    const int p = (int)(i / half);
    const double inv = pow(base, -2.0 * j / (2.0 * half));
    const double th = (double)p * inv;
    t[i] = make_float2((float)cos(th), (float)sin(th));
}

// Copy with element conversion (embedding / gains into the library's own copy).
template <typename ST, typename DT>
__global__ void __launch_bounds__(256) convert_kernel(const ST* s, DT* d, size_t n) {
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) d[i] = from_f32<DT>(to_f32<ST>(s[i]));
}

// Per-row key limit of refreshed rows: end of the row's block, capped at the prefix.
__global__ void refresh_limits_kernel(const int* pos, int n, int prompt_len, int block, int prefix_len,
                                      int* lim) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const int p = pos[i];
    int e = (p < prompt_len) ? prompt_len : prompt_len + block * (1 + (p - prompt_len) / block);
    lim[i] = min(e, prefix_len);
}

// Draft acceptance when a block becomes current: a masked position whose draft
// record equals this step's prediction with conf >= theta is committed; the
// accepted positions are written in ascending order (ballot compaction).
__global__ void __launch_bounds__(1024)
accept_drafts_kernel(const float* conf, const int* id, const int* draft, int* tok, uint8_t* mask, int n, float theta,
                     int* accepted, int* n_accepted) {
    __shared__ int wsum[16];
    const int i = threadIdx.x;
    bool a = false;
    if (i < n && mask[i] == 1) {
        const int dv = draft[i];
        a = dv >= 0 && id[i] == dv && conf[i] >= theta;
    }
    if (a) {
        tok[i] = id[i];
        mask[i] = 0;
    }
    const unsigned long long bal = __ballot(a);
    const int lane = i & 63, w = i >> 6;
    if (lane == 0) wsum[w] = __popcll(bal);
    __syncthreads();
    int off = 0;
    for (int j = 0; j < w; ++j) off += wsum[j];
    if (a && accepted != nullptr) accepted[off + __popcll(bal & ((1ull << lane) - 1ull))] = i;
    if (i == 0 && n_accepted != nullptr) {
        int t = 0;
        for (int j = 0; j < (int)(blockDim.x >> 6); ++j) t += wsum[j];
        *n_accepted = t;
    }
}

// Draft records: this step's prediction for masked positions, -1 elsewhere.
__global__ void record_drafts_kernel(const int* id, const uint8_t* mask, int* draft, int n) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) draft[i] = mask[i] == 1 ? id[i] : -1;
}

// Rows of a merged pass (refresh, append and step in one forward): rows [0, n_ref)
// are revised prefix positions (keys up to the end of their block, capped at P),
// rows [n_ref, n_ref + n_blk) the completed block at P.. (keys [0, P + n_blk)),
// the last W rows the window at P + n_blk.. (keys [0, P + n_blk + W), mask kept).
// need: the rows whose (id, conf) is asked for (refresh rows if ref_out, window
// rows if win_out; the appended block never).
__global__ void merged_rows_kernel(const int* ref_pos, const int* ref_id, int n_ref, const int* blk, int n_blk,
                                   const int* tok, const uint8_t* mask, int W, int P, int prompt_len, int block,
                                   int ref_out, int win_out, int* otok, uint8_t* omask, int* opos, int* olim,
                                   uint8_t* oneed) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n_ref + n_blk + W) return;
    int t, p, l;
    uint8_t mk = 0;
    if (i < n_ref) {
        p = ref_pos[i];
        t = ref_id[i];
        const int e = (p < prompt_len) ? prompt_len : prompt_len + block * (1 + (p - prompt_len) / block);
        l = min(e, P);
    } else if (i < n_ref + n_blk) {
        const int j = i - n_ref;
        t = blk[j];
        p = P + j;
        l = P + n_blk;
    } else {
        const int j = i - n_ref - n_blk;
        t = tok[j];
        mk = mask ? mask[j] : (uint8_t)0;
        p = P + n_blk + j;
        l = P + n_blk + W;
    }
    otok[i] = t;
    omask[i] = mk;
    opos[i] = p;
    olim[i] = l;
    oneed[i] = (uint8_t)(i < n_ref ? ref_out : (i < n_ref + n_blk ? 0 : win_out));
}

// Outputs of a merged pass: the refresh rows' and the window rows' (id, conf).
__global__ void merged_out_kernel(const int* oid, const float* oconf, int n_ref, int n_blk, int W, int* ref_id,
                                  float* ref_conf, int* out_id, float* out_conf) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n_ref && ref_id) {
        ref_id[i] = oid[i];
        ref_conf[i] = oconf[i];
    } else if (i >= n_ref + n_blk && i < n_ref + n_blk + W && out_id) {
        out_id[i - n_ref - n_blk] = oid[i];
        out_conf[i - n_ref - n_blk] = oconf[i];
    }
}

}  // namespace dllm
