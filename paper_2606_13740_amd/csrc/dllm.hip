// libdllm: host runtime and C ABI of the gfx950 denoising-step library.
//
// One denoising step (a window of W <= 64 rows over a prefix cache) is, per
// layer: fused RMSNorm+QKV+RoPE GEMM (K/V straight into the cache), window-vs-
// prefix attention (+ split merge), O projection + residual, fused
// RMSNorm+gate/up+SwiGLU GEMM, down projection + residual; then the final norm +
// LM head fused with the (max, argmax, sum exp) reduction and its merge.  Every
// launch is on the caller's stream; nothing is synchronised on the step path.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <type_traits>
#include <vector>

#include "../../include/dllm.h"
#include "attention.hpp"
#include "common.hpp"
#include "gemm.hpp"
#include "gemm_tiled.hpp"
#include "kernels.hpp"

using namespace dllm;

namespace {

thread_local std::string g_last_error;

int fail(int code, const std::string& msg) {
    g_last_error = msg;
    return code;
}

#define HIP_TRY(expr)                                                                           \
    do {                                                                                        \
        hipError_t _e = (expr);                                                                 \
        if (_e != hipSuccess)                                                                   \
            return fail(DLLM_E_HIP, std::string(#expr) + ": " + hipGetErrorString(_e));        \
    } while (0)

inline int ceil_div(long a, long b) { return (int)((a + b - 1) / b); }
inline long round_up(long a, long b) { return (a + b - 1) / b * b; }

// One packed GEMM operand.
struct PackedW {
    void* w = nullptr;      // chunks
    float* scale = nullptr; // per packed row (int8) or nullptr
    uint16_t* qs = nullptr; // Q4_0 block scales (fp16) or nullptr
    size_t qs_bytes = 0;
    int N = 0;              // real rows
    int K = 0;              // real columns
    int n_tiles = 0;
    int KCw = 0;
    size_t bytes = 0;
};

struct LayerW {
    PackedW qkv, o, gu, down;
    float* g1 = nullptr;
    float* g2 = nullptr;
    float* bqkv = nullptr;   // Q/K/V biases in packed-row order, or nullptr
};

struct Workspace {
    void* block = nullptr;   // the one device allocation the buffers below are carved from
    int rows = 0;            // token rows (multiple of 64)
    int wrows = 0;           // window rows for LM / attention partials (multiple of 64)
    float* x = nullptr;      // [rows][d]
    void* xg = nullptr;      // fragments, K = d
    void* q = nullptr;       // [rows][d] act type
    void* of = nullptr;      // fragments, K = d (attention output)
    void* af = nullptr;      // fragments, K = d_ff
    int* pos = nullptr;      // [rows]
    int* lim = nullptr;      // [rows]
    LmPartial* lm = nullptr; // [n_lm_wg][wrows]
    float* part = nullptr;   // split-K partials [KS][rows][d]
    size_t part_floats = 0;
    float* opart = nullptr;  // [MAX_SPLIT][wrows][H][Dh]
    float* mlpart = nullptr; // [MAX_SPLIT][wrows][H][2]
    float* ssq = nullptr;    // [d / 16][rows] sum-of-squares partials of a folded RMSNorm
    int* slot = nullptr;     // [rows] LM-head slot of each row (selective logits skipping)
    int ssq_ld = 0;          // partials per row of ssq (a multiple of 64)
    size_t xg_bytes = 0, of_bytes = 0, af_bytes = 0;   // allocated fragment-buffer sizes
    int* tok = nullptr;      // [rows] ids of a merged pass
    uint8_t* msk = nullptr;  // [rows] mask flags of a merged pass
    int* oid = nullptr;      // [rows] argmax ids of a merged pass
    float* oconf = nullptr;  // [rows] confidences of a merged pass
    uint8_t* need = nullptr; // [rows] LM-head row flags of a merged pass
};

constexpr int MAX_SPLIT = 16;
// Windows of <= 64 rows: most 32-key blocks one attention key group streams before the
// key range is split across workgroups (and merged by a separate launch).
#ifndef ATTN_ROUNDS
#define ATTN_ROUNDS 3
#endif
constexpr int ATTN_KEYGROUP_BLOCKS = 48;
constexpr int RES_SPLIT = 8;     // most K slices of the O / down projections for windows of <= 64 rows

}  // namespace

struct dllm_model {
    dllm_config cfg;
    int wt = 0;              // WT_F32 / WT_BF16 / WT_I8
    bool xf32 = false;       // activations in fp32
    size_t kv_elem = 4;      // bytes per cached K or V value (fp32 or fp16)
    int KCx_d = 0, KCx_f = 0;
    int Hkv = 0, dkv = 0;    // K/V heads and K (or V) rows per layer
    std::vector<LayerW> layers;
    PackedW lm;
    void* embed = nullptr;
    float* gf = nullptr;
    float2* rope = nullptr;
    void* wpool = nullptr;   // packed weights of every matrix
    float* spool = nullptr;  // int8 scales
    uint16_t* qpool = nullptr;  // Q4_0 scales
    float* gpool = nullptr;  // norm gains
    float* bpool = nullptr;  // Q/K/V biases
    Workspace ws;
    int n_lm_wg = 1;
    // probe
    int probe_class = -1;
    int probe_max = 0;
    int probe_n = 0;
    std::vector<hipEvent_t> ev_b, ev_e;
};

struct dllm_kv {
    const dllm_model* model;
    void* buf;
    size_t bytes;
    int capacity;
    int Cs;
    int prefix_len;
    int prompt_len;
};

namespace {

// ---------------------------------------------------------------------------
// Launch configuration of the weight-streaming GEMMs
// ---------------------------------------------------------------------------

enum GemmKind { G_QKV = 0, G_RES = 1, G_GU = 2, G_LM = 3 };

int pick_MT(int M) {
    if (M <= 16) return 1;
    if (M <= 32) return 2;
    if (M <= 48) return 3;
    return 4;
}

// Decompositions (measured on MI355X at the LLaDA-8B shapes, weights rotated
// through >1 GB so that HBM is streamed):
//   QKV    3 row tiles per workgroup, K split over 8 waves          (4.3 TB/s)
//   gate/up 6 row tiles per workgroup, K split over 8 waves         (5.2 TB/s)
//   LM head 4 waves x 8 row tiles, each wave streams the whole K    (6.3 TB/s)
//   O/down 4 row tiles, K split over 8 waves x 4 workgroups (split-K) + reduction
// These are template shapes; a launch may give each wave group fewer row tiles
// (tpg) and fewer split-K slices (ks).  Every workgroup of these layouts holds a
// whole CU (8 waves at ~200 VGPRs, or 100+ KiB of LDS), so a launch of more than
// 256 workgroups runs in rounds: (tpg, ks) is chosen to minimise the busiest CU's
// share, rounds x (tpg / ks + 1) row tiles of full K, the 1 standing for a
// workgroup's fixed cost (start-up, K-slice reduction, epilogue); this picks the
// layouts above at the LLaDA-8B widths (256 or 247 workgroups) and e.g. 5 tiles
// per wave group for the Dream-7B LM head (its gate/up takes the 10-tile template
// below).  Small models (fewer row tiles than the thresholds below) use one tile per
// 4-wave workgroup.
struct Decomp {
    bool small;   // 1 tile per workgroup of 4 waves, K over the waves
    int tpg;      // row tiles per wave group
    int ks;       // split-K slices (residual projections)
    bool wide = false;   // long prompts: whole-K waves of 8 row tiles (WIDE_TILES)
    bool tiled = false;  // 256+ rows: gemm_tiled_kernel (LDS-staged tiles; tiled_layout)
};

constexpr int N_CU = 256;
// A second gate/up template for widths that fill the chip in one round only with more
// than 6 row tiles per wave group (Dream-7B: 2368 row tiles, 10 per group in 237
// workgroups: 46.2 against 53.1 us for 5 per group in two rounds).  It runs 2 weight
// stages where the 6-tile template runs 3, so the LLaDA-8B widths keep the 6-tile one.
constexpr int GU_WIDE_TILES = 10;

// bf16 and int8 GEMMs over 256 or more token rows (prompts, wide windows) except the
// LM head run the LDS-tiled kernel when it gives the chip at least TILED_MIN_WG
// workgroups: every weight and activation chunk is fetched once per 256-row x 256-token
// tile (int8: 128 tokens) and shared by the workgroup's waves (LLaDA-8B bf16 at 512
// rows: gate/up 201 against 276 us, down 107 against 173; at 4096 rows gate/up 1063
// against 2825, QKV 823 against 1735).  With fewer workgroups the streaming layouts
// win (QKV at 512 rows, 96 tiles: 238 against 201 us; every GEMM of a 256-row
// window), except that bf16 QKV of up to 682 rows splits K in two when that reaches
// TILED_MIN_WG (tiled_ks; LLaDA-8B at 512 rows: 192 workgroups, 192 -> 117 us per
// layer with the split_epilogue_kernel finish).  Models below the streaming
// layouts' thresholds (test sizes) take it whenever it applies: it accepts any row
// and token tile counts (ragged tiles are clamped).  The residual projections split
// K until the chip holds ~256 workgroups (O/down at 512 rows: 32 tiles x 8 slices);
// their partial buffer holds min(8 x rows, 4096) rows.  int8 weights take it for QKV
// only: every wave widens the int8 chunks it reads from LDS, four times over per
// chunk, which makes the larger projections VALU-bound (4096 rows: QKV 1460 -> 1118
// us, but gate/up 1799 -> 1984 and down 855 -> 1086 against the whole-K layout).
constexpr int TILED_MIN_WG = 192;
bool tiled_layout(GemmKind k, int wt, int Mc) {
    return Mc >= 256 && ((wt == WT_BF16 && k != G_LM) || (wt == WT_I8 && k == G_QKV));
}
// token tiles per workgroup of the tiled kernel
int tiled_tt(int wt) { return wt == WT_I8 ? TiledShape<WT_I8>::TT : TiledShape<WT_BF16>::TT; }
int tiled_ks(GemmKind k, int wt, int n_tiles, int Mc) {
    const long wgs = (long)ceil_div(n_tiles, 16) * ceil_div(Mc / 16, tiled_tt(wt));
    if (k == G_QKV) {
        // bf16 QKV of short prompts: two K slices when one leaves fewer than
        // TILED_MIN_WG workgroups and two fit the chip (LLaDA-8B at 512 rows: 96 -> 192),
        // finished by split_epilogue_kernel; two slices of an output at most 3 d wide
        // fit the partial buffer up to 682 rows
        return (wt == WT_BF16 && wgs < TILED_MIN_WG && 2 * wgs <= N_CU && 6 * Mc <= 4096) ? 2 : 1;
    }
    if (k != G_RES) return 1;
    int ks = 1;
    while (ks < 8 && wgs * ks * 2 <= N_CU && (long)ks * 2 * Mc <= 4096) ks *= 2;
    return ks;
}

// More than 8 token blocks of 64 rows (prompts past 512 tokens, bf16 / int8
// weights), gate/up and O/down: each wave takes 8 row tiles over the whole K range,
// 4 row groups per workgroup sharing one token block.  The K-sliced layouts
// re-stream every row group's weights once per token block and reach ~290 TFLOP/s
// there; this one holds 8 x 4 tiles of accumulators per wave (LLaDA-8B, int8, 4096
// rows: gate/up 1980 -> 1817 us, down 1156 -> 859 us, O 462 -> 371 us).  QKV keeps
// its layout: with 2 row groups per workgroup (its RoPE staging needs the LDS) the
// epilogue over 128 rows x 64 tokens on 128 threads made it slower (1521 -> 1688 us).
// Up to 8 blocks the K-sliced layouts with the XCD-aware block order are faster.
constexpr int WIDE_TILES = 8;
bool wide_layout(GemmKind k, int wt, int gy) {
    return gy > 8 && (k == G_GU || k == G_RES) && (wt == WT_BF16 || wt == WT_I8);
}

// Row tiles per wave group of each template at mt token tiles.  Q4_0 exceptions:
// the LM head takes 4, since at 8 its code pipeline, activations and 16
// accumulators per token tile need more than 256 registers and leave one wave per
// SIMD (LLaDA-8B vocabulary at 32 rows: 119 against 144 us per launch); the
// gate/up and the split-K projections take 3 past 2 token tiles, where 6 (gate/up)
// or 4 (down: 47 registers at 4 token tiles) would spill.  bf16 split-K projections
// up to 2 token tiles (the down projection of windows of <= 32 rows) take 8 tiles
// over 8 K slices instead of 4 over 4: the same 256 workgroups, but every workgroup
// re-reads the hi/lo activation operand of its K slice through L2, so twice the
// rows per workgroup halve that traffic (LLaDA-8B down at 32 rows: 28.6 -> 26.8 us
// per launch with the reduction, against twice the partial sums).
constexpr int template_fw(GemmKind k, int wt, int mt) {
    if (wt == WT_Q4 && (k == G_GU || k == G_RES) && mt >= 3) return 3;
    if (wt == WT_BF16 && k == G_RES && mt <= 2) return 8;
    return k == G_QKV ? 3 : (k == G_GU ? 6 : (k == G_LM ? (wt == WT_Q4 ? 4 : 8) : 4));
}
int template_nwn(GemmKind k) { return k == G_LM ? 4 : 1; }

Decomp decomp(GemmKind k, int wt, int n_tiles, int Mc, int gy) {
    const int min_tiles = (k == G_QKV || k == G_RES) ? 128 : (k == G_GU ? 256 : 512);
    if (tiled_layout(k, wt, Mc)) {
        const int ks = tiled_ks(k, wt, n_tiles, Mc);
        const long wgs = (long)ceil_div(n_tiles, 16) * ceil_div(Mc / 16, tiled_tt(wt)) * ks;
        if (n_tiles < min_tiles || wgs >= TILED_MIN_WG) return Decomp{false, 16, ks, false, true};
    }
    if (n_tiles < min_tiles) return Decomp{true, 1, 1};
    if (wide_layout(k, wt, gy)) return Decomp{false, WIDE_TILES, 1, true};
    const int fw = template_fw(k, wt, Mc / (16 * gy)), nwn = template_nwn(k);
    Decomp best{false, 1, 1};
    double best_load = 1e30;
    // bf16 gate/up up to 2 token tiles may also take the 10-tile template
    // (GU_WIDE_TILES), for widths whose row tiles would need two rounds at 6
    const int mt = Mc / (16 * gy);
    const int fw_max = (k == G_GU && wt == WT_BF16 && mt <= 2) ? GU_WIDE_TILES : fw;
    for (int tpg = fw_max; tpg >= 1; --tpg) {
        for (int ks = (k == G_RES && Mc <= 64) ? RES_SPLIT : 1; ks >= 1; ks >>= 1) {
            const long wgs = (long)ceil_div(ceil_div(n_tiles, tpg), nwn) * ks * gy;
            // busiest CU: rounds x (its tiles of full K + a workgroup's fixed cost, about
            // one tile).  Every template slot's MFMAs run whether or not the group fills
            // it, so past 2 token tiles a group costs at least half the template.
            const double work = Mc > 32 ? std::max<double>(tpg, fw / 2.0) : (double)tpg;
            const double load = (double)ceil_div(wgs, N_CU) * (work / ks + 1.0);
            if (load < best_load - 1e-9) { best_load = load; best = Decomp{false, tpg, ks}; }
        }
    }
    return best;
}

template <int WT, int FW, int NWn, int NWk, int MT, class Epi>
void launch_gemm_inst(const GemmArgs& g, const Epi& epi, int n_tiles, int KS, int gy, hipStream_t s) {
    dim3 grid(ceil_div(ceil_div(n_tiles, g.tpg), NWn), KS, gy);
    hipLaunchKernelGGL((gemm_kernel<WT, FW, NWn, NWk, MT, Epi>), grid, dim3(NWn * NWk * 64), 0, s, g, epi);
}

// Row tiles of kind KIND_FW's template at mt token tiles; KIND_FW < 0 is the
// small-model layout (one tile).
template <int WT, int KIND_FW>
constexpr int fw_of(int mt) { return KIND_FW < 0 ? 1 : template_fw((GemmKind)KIND_FW, WT, mt); }

template <int WT, int KIND_FW, int NWn, int NWk, class Epi>
int launch_gemm_mt(int MT, const GemmArgs& g, const Epi& epi, int n_tiles, int KS, int gy, hipStream_t s) {
    constexpr auto fw = fw_of<WT, KIND_FW>;
    if (MT < 1 || MT > 4) return fail(DLLM_E_UNIMPL, "unsupported token tile count");
    if (g.tpg < 1 || g.tpg > fw(MT)) return fail(DLLM_E_INVAL, "internal: row tiles per group outside the template");
    switch (MT) {
        case 1: launch_gemm_inst<WT, fw(1), NWn, NWk, 1>(g, epi, n_tiles, KS, gy, s); break;
        case 2: launch_gemm_inst<WT, fw(2), NWn, NWk, 2>(g, epi, n_tiles, KS, gy, s); break;
        case 3: launch_gemm_inst<WT, fw(3), NWn, NWk, 3>(g, epi, n_tiles, KS, gy, s); break;
        default: launch_gemm_inst<WT, fw(4), NWn, NWk, 4>(g, epi, n_tiles, KS, gy, s); break;
    }
    return DLLM_OK;
}

// Number of row groups (LM-head partial records) a launch writes.
int row_groups(const Decomp& dc, int n_tiles) { return ceil_div(n_tiles, dc.tpg); }

template <int WT, GemmKind KIND, class Epi>
int launch_gemm(const Decomp& dc, int n_tiles, int MT, const GemmArgs& g0, const Epi& epi, int gy, hipStream_t s,
                float* part = nullptr, size_t part_floats = 0) {
    GemmArgs g = g0;
    g.tpg = dc.tpg;
    if constexpr ((WT == WT_BF16 && KIND != G_LM) || (WT == WT_I8 && KIND == G_QKV)) {
        if (dc.tiled) {
            using TS = TiledShape<WT>;
            const int Mc = gy * MT * 16;
            if (Mc % 64 != 0) return fail(DLLM_E_INVAL, "internal: tiled GEMM needs 64-row blocks");
            dim3 grid(ceil_div(n_tiles, TS::RT), dc.ks, ceil_div(Mc / 16, TS::TT));
            if constexpr (KIND == G_QKV && WT == WT_BF16) {
                if (dc.ks > 1) {
                    // K slices into partial sums, then split_epilogue_kernel sums them and
                    // runs the QKV epilogue (the bias goes in once, after the sum)
                    const int N = n_tiles * 16;
                    if (part == nullptr || (size_t)dc.ks * Mc * N > part_floats)
                        return fail(DLLM_E_INVAL, "internal: split-K buffer too small");
                    GemmArgs gp = g0;
                    gp.bias = nullptr;
                    const EpiPartial ep{part, N, Mc};
                    hipLaunchKernelGGL((gemm_tiled_kernel<WT, EpiPartial>), grid, dim3(512), 0, s, gp, ep, Mc / 16);
                    hipLaunchKernelGGL((split_epilogue_kernel<Epi>), dim3(ceil_div(n_tiles, 16), ceil_div(Mc / 16, 4)),
                                       dim3(256), 0, s, (const float*)part, dc.ks, Mc, N, n_tiles, Mc / 16, g0.bias,
                                       epi);
                    return DLLM_OK;
                }
            }
            hipLaunchKernelGGL((gemm_tiled_kernel<WT, Epi>), grid, dim3(512), 0, s, g0, epi, Mc / 16);
            return DLLM_OK;
        }
    }
    if (dc.small) return launch_gemm_mt<WT, -1, 1, 4>(MT, g, epi, n_tiles, dc.ks, gy, s);
    if constexpr (KIND == G_GU && WT == WT_BF16) {
        if (g.tpg > template_fw(G_GU, WT, MT)) {
            if (g.tpg > GU_WIDE_TILES || MT > 2) return fail(DLLM_E_INVAL, "internal: gate/up tiles outside the templates");
            if (MT == 1) launch_gemm_inst<WT, GU_WIDE_TILES, 1, 8, 1>(g, epi, n_tiles, 1, gy, s);
            else launch_gemm_inst<WT, GU_WIDE_TILES, 1, 8, 2>(g, epi, n_tiles, 1, gy, s);
            return DLLM_OK;
        }
    }
    if constexpr ((WT == WT_BF16 || WT == WT_I8) && (KIND == G_GU || KIND == G_RES)) {
        if (dc.wide) {
            if (MT != 4 || g.tpg != WIDE_TILES) return fail(DLLM_E_INVAL, "internal: wide layout needs 64-row blocks");
            launch_gemm_inst<WT, WIDE_TILES, 4, 1, 4>(g, epi, n_tiles, 1, gy, s);
            return DLLM_OK;
        }
    }
    if constexpr (KIND == G_LM) return launch_gemm_mt<WT, G_LM, 4, 1>(MT, g, epi, n_tiles, 1, gy, s);
    else return launch_gemm_mt<WT, KIND, 1, 8>(MT, g, epi, n_tiles, KIND == G_RES ? dc.ks : 1, gy, s);
}

// ---------------------------------------------------------------------------
// Probe
// ---------------------------------------------------------------------------

struct ProbeScope {
    dllm_model* m;
    hipStream_t s;
    bool on;
    ProbeScope(dllm_model* m_, int cls, hipStream_t s_) : m(m_), s(s_) {
        on = (m->probe_class == cls && m->probe_n < m->probe_max);
        if (on) (void)hipEventRecord(m->ev_b[m->probe_n], s);
    }
    ~ProbeScope() {
        if (on) {
            (void)hipEventRecord(m->ev_e[m->probe_n], s);
            ++m->probe_n;
        }
    }
};

// ---------------------------------------------------------------------------
// Workspace
// ---------------------------------------------------------------------------

void free_ws(Workspace& w) {
    if (w.block) (void)hipFree(w.block);
    w = Workspace{};
}

int alloc_zero(void** p, size_t bytes) {
    if (hipMalloc(p, std::max<size_t>(bytes, 256)) != hipSuccess) {
        *p = nullptr;
        return fail(DLLM_E_NOMEM, "device allocation of " + std::to_string(bytes) + " bytes failed");
    }
    HIP_TRY(hipMemset(*p, 0, std::max<size_t>(bytes, 256)));
    return DLLM_OK;
}

// The buffers of a workspace for `rows` token rows (a multiple of 64), LM-head and
// attention partials for `wrows` rows, and `part_floats` split-K partials, laid out
// one after another (256-byte aligned) from `base`.  Returns the bytes they take; with
// base == nullptr only the size is computed.  Every user of a workspace (the model's
// own, grown on demand, and the no-allocation step's static scratch) is carved here.
size_t ws_carve(const dllm_model* m, int rows, int wrows, size_t part_floats, char* base, Workspace* w);

// Split-K partials: 4 slices of the window rows (streaming layouts), or up to 8 slices
// of 256+ token rows (tiled layout), at most 4096 rows.
size_t part_floats_for(const dllm_model* m, int rows, int wrows) {
    return (size_t)std::max({RES_SPLIT * wrows, rows, std::min(8 * rows, 4096)}) * m->cfg.d_model;
}

int ensure_ws(dllm_model* m, int rows_needed) {
    const dllm_config& c = m->cfg;
    const int rows = (int)round_up(std::max(rows_needed, 1), 64);
    if (m->ws.rows >= rows && m->ws.block) return DLLM_OK;
    HIP_TRY(hipDeviceSynchronize());
    free_ws(m->ws);
    const int wrows = (int)round_up(c.max_window, 64);
    const size_t part_floats = part_floats_for(m, rows, wrows);
    const size_t bytes = ws_carve(m, rows, wrows, part_floats, nullptr, nullptr);
    void* blk = nullptr;
    int rc = alloc_zero(&blk, bytes);
    if (rc) return rc;
    ws_carve(m, rows, wrows, part_floats, (char*)blk, &m->ws);
    m->ws.block = blk;
    return DLLM_OK;
}

// ---------------------------------------------------------------------------
// Weight prepacking
// ---------------------------------------------------------------------------

size_t ws_carve(const dllm_model* m, int rows, int wrows, size_t part_floats, char* base, Workspace* w) {
    const dllm_config& c = m->cfg;
    const size_t d = c.d_model;
    const size_t xchunk = m->xf32 ? 1024 : 2048;   // an activation chunk: fp32, or bf16 hi + lo
    const size_t xg_bytes = (size_t)(rows / 16) * m->KCx_d * xchunk;
    const size_t af_bytes = (size_t)(rows / 16) * m->KCx_f * xchunk;
    size_t off = 0;
    auto take = [&](auto*& ptr, size_t bytes) {
        if (base) ptr = (std::remove_reference_t<decltype(ptr)>)(base + off);
        off += round_up((long)std::max<size_t>(bytes, 1), 256);
    };
    Workspace tmp;
    Workspace& v = w ? *w : tmp;
    v.rows = rows;
    v.wrows = wrows;
    v.xg_bytes = v.of_bytes = xg_bytes;
    v.af_bytes = af_bytes;
    v.part_floats = part_floats;
    take(v.x, (size_t)rows * d * 4);
    take(v.xg, xg_bytes);
    take(v.q, (size_t)rows * d * 4);   // fp32, or bf16 hi and lo planes
    take(v.of, xg_bytes);
    take(v.af, af_bytes);
    take(v.pos, (size_t)rows * 4);
    take(v.lim, (size_t)rows * 4);
    take(v.lm, (size_t)m->n_lm_wg * wrows * sizeof(LmPartial));
    take(v.part, part_floats * 4);
    take(v.opart, (size_t)MAX_SPLIT * wrows * d * 4);
    take(v.mlpart, (size_t)MAX_SPLIT * wrows * c.n_heads * 2 * 4);
    v.ssq_ld = (int)round_up(ceil_div(c.d_model, 16), 64);
    take(v.ssq, (size_t)v.ssq_ld * rows * 4);
    take(v.slot, (size_t)rows * 4);
    take(v.tok, (size_t)rows * 4);
    take(v.msk, (size_t)rows);
    take(v.oid, (size_t)rows * 4);
    take(v.oconf, (size_t)rows * 4);
    take(v.need, (size_t)rows);
    return off;
}

int kc_of(int wt) { return wt == WT_F32 ? 16 : (wt == WT_BF16 ? 32 : 64); }

void plan_packed(PackedW& p, int wt, int N, int K) {
    p.N = N;
    p.K = K;
    p.n_tiles = ceil_div(N, 16);
    p.KCw = ceil_div(K, kc_of(wt));
    p.bytes = (size_t)p.n_tiles * p.KCw * (wt == WT_Q4 ? 512 : 1024);
    p.qs_bytes = (wt == WT_Q4) ? (size_t)p.n_tiles * p.KCw * 64 : 0;   // 16 rows x 2 blocks x fp16
}

template <typename ST>
int pack_one(dllm_model* m, PackedW& p, const PackSrc& src, hipStream_t s) {
    const size_t units = (size_t)p.n_tiles * p.KCw * 64;
    const int blocks = ceil_div((long)units, 256);
    if (m->wt == WT_Q4) {
        hipLaunchKernelGGL((pack_q4_kernel<ST>), dim3(blocks), dim3(256), 0, s, src, p.n_tiles, p.KCw, (u32x2_t*)p.w,
                           p.qs);
    } else if (m->wt == WT_I8) {
        hipLaunchKernelGGL((row_scale_kernel<ST>), dim3(p.n_tiles * 16), dim3(256), 0, s, src, p.n_tiles * 16, p.scale);
        hipLaunchKernelGGL((pack_kernel<WT_I8, ST>), dim3(blocks), dim3(256), 0, s, src, p.n_tiles, p.KCw,
                           (u32x4_t*)p.w, (const float*)p.scale);
    } else if (m->wt == WT_BF16) {
        hipLaunchKernelGGL((pack_kernel<WT_BF16, ST>), dim3(blocks), dim3(256), 0, s, src, p.n_tiles, p.KCw,
                           (u32x4_t*)p.w, (const float*)nullptr);
    } else {
        hipLaunchKernelGGL((pack_kernel<WT_F32, ST>), dim3(blocks), dim3(256), 0, s, src, p.n_tiles, p.KCw,
                           (u32x4_t*)p.w, (const float*)nullptr);
    }
    HIP_TRY(hipGetLastError());
    return DLLM_OK;
}

int validate_config(const dllm_config* c) {
    if (!c) return fail(DLLM_E_INVAL, "config is NULL");
    if (c->n_layers < 1 || c->d_model < 1 || c->n_heads < 1 || c->head_dim < 1 || c->d_ff < 1 || c->vocab < 2)
        return fail(DLLM_E_INVAL, "shape fields must be positive (vocab >= 2)");
    if (c->n_heads * c->head_dim != c->d_model) return fail(DLLM_E_INVAL, "d_model != n_heads * head_dim");
    if (c->mask_id < 0 || c->mask_id >= c->vocab) return fail(DLLM_E_INVAL, "mask_id out of range");
    if (c->block < 1) return fail(DLLM_E_INVAL, "block must be >= 1");
    if (c->max_window < 1 || c->max_window > 256) return fail(DLLM_E_INVAL, "max_window must be in [1, 256]");
    if (c->max_pos < 1) return fail(DLLM_E_INVAL, "max_pos must be >= 1");
    if (!(c->eps > 0.f) || !(c->rope_base > 1.f)) return fail(DLLM_E_INVAL, "eps must be > 0 and rope_base > 1");
    if (c->dtype != DLLM_F32 && c->dtype != DLLM_BF16 && c->dtype != DLLM_W8 && c->dtype != DLLM_Q4)
        return fail(DLLM_E_DTYPE, "dtype must be DLLM_F32, DLLM_BF16, DLLM_W8 or DLLM_Q4");
    if (c->dtype == DLLM_F32) {
        if (c->head_dim != 32 && c->head_dim != 64 && c->head_dim != 128)
            return fail(DLLM_E_DTYPE, "fp32 models need head_dim 32, 64 or 128");
    } else if (c->head_dim != 64 && c->head_dim != 128) {
        return fail(DLLM_E_DTYPE, "bf16 / int8 / Q4_0 models need head_dim 64 or 128");
    }
    if (c->d_model % 32 != 0) return fail(DLLM_E_DTYPE, "d_model must be a multiple of 32");
    if (c->d_model > 4 * ROW_NT * ROW_VPT) return fail(DLLM_E_DTYPE, "d_model must be <= 8192");
    if (c->d_ff % 8 != 0) return fail(DLLM_E_DTYPE, "d_ff must be a multiple of 8");
    if (c->n_kv_heads < 0 || c->n_kv_heads > c->n_heads || (c->n_kv_heads > 0 && c->n_heads % c->n_kv_heads != 0))
        return fail(DLLM_E_INVAL, "n_kv_heads must be 0 or divide n_heads");
    if (c->qkv_bias != 0 && c->qkv_bias != 1) return fail(DLLM_E_INVAL, "qkv_bias must be 0 or 1");
    return DLLM_OK;
}

// ---------------------------------------------------------------------------
// The forward over a set of rows
// ---------------------------------------------------------------------------

struct FwdArgs {
    int M;                    // rows
    const int* tok;           // ids
    const uint8_t* mask;      // nullable
    int pos_base;             // row m at pos_base + m unless pos
    const int* pos;           // device positions or nullptr
    int T;                    // key count for rows without own limit
    const int* lim;           // per-row limits or nullptr
    int n_layers;             // layers to run
    bool lm;
    float* logits;            // debug logits or nullptr
    int* out_id;
    float* out_conf;
    float* xout;              // residual copy or nullptr
    bool sel;                 // LM head over selected rows only (selective logits skipping)
    const uint8_t* need;      // device row flags (nullable: every row) when sel
    int n_sel;                // at most this many flagged rows get an LM output
    int replay = -1;          // >= 0: only launch this kernel class, n_replay times (timing)
    int n_replay = 0;
    Workspace* ws = nullptr;  // a caller-provided workspace (no growth), else the model's
};

// O / down projection: split-K GEMM into partials, then the reduction that adds
// them to the residual and prepares the next RMSNorm's operand and partial sums.
template <int WT, bool XF32>
int residual_proj(dllm_model* m, Workspace& w, const PackedW& W, const void* X, const float* gnext, int M, int Mc,
                  int MT, int gy, hipStream_t s, bool sel = false, const uint8_t* need = nullptr, int n_sel = 0) {
    const int d = m->cfg.d_model;
    const Decomp dc = decomp(G_RES, WT, W.n_tiles, Mc, gy);
    const int KS = dc.ks;
    if ((size_t)KS * Mc * d > w.part_floats) return fail(DLLM_E_INVAL, "internal: split-K buffer too small");
    GemmArgs g{W.w, W.scale, X, W.KCw, W.KCw * WTraits<WT>::XPER, W.n_tiles};
    g.qs = W.qs;
    EpiPartial e{w.part, d, Mc};
    int rc = launch_gemm<WT, G_RES>(dc, W.n_tiles, MT, g, e, gy, s);
    if (rc) return rc;
#define RRED(KS_)                                                                                              \
    hipLaunchKernelGGL((residual_reduce_kernel<XF32, KS_>), dim3(Mc), dim3(ROW_NT), 0, s, (const float*)w.part, Mc, \
                       d, M, m->cfg.eps, w.x, gnext, w.xg, m->KCx_d, sel, need, n_sel)
    switch (KS) {
        case 1: RRED(1); break;
        case 2: RRED(2); break;
        case 4: RRED(4); break;
        case 8: RRED(8); break;
        default: return fail(DLLM_E_INVAL, "internal: K slices of a residual projection not 1, 2, 4 or 8");
    }
#undef RRED
    return DLLM_OK;
}

// O / down projection of a window of <= 64 rows with the next RMSNorm folded into
// the consumer: the whole K range per workgroup (one row tile, 8 waves over K, no
// split-K partials and no reduction launch); the epilogue updates x, writes the next
// GEMM's operand x * g_next and one sum-of-squares partial per row tile and token.
template <int WT, bool XF32>
int residual_proj_fused(dllm_model* m, Workspace& w, const PackedW& W, const void* X, const float* gnext, int M,
                        int MT, hipStream_t s, const int* slot = nullptr) {
    GemmArgs g{W.w, W.scale, X, W.KCw, W.KCw * WTraits<WT>::XPER, W.n_tiles};
    g.qs = W.qs;
    g.tpg = 1;
    EpiResidual<XF32> e{w.x, m->cfg.d_model, M, gnext, w.xg, m->KCx_d, w.ssq, w.ssq_ld, slot};
    switch (MT) {
        case 1: launch_gemm_inst<WT, 1, 1, 8, 1>(g, e, W.n_tiles, 1, 1, s); break;
        case 2: launch_gemm_inst<WT, 1, 1, 8, 2>(g, e, W.n_tiles, 1, 1, s); break;
        case 3: launch_gemm_inst<WT, 1, 1, 8, 3>(g, e, W.n_tiles, 1, 1, s); break;
        case 4: launch_gemm_inst<WT, 1, 1, 8, 4>(g, e, W.n_tiles, 1, 1, s); break;
        default: return fail(DLLM_E_UNIMPL, "unsupported token tile count");
    }
    return DLLM_OK;
}

// The consumer side of a folded RMSNorm: the GEMM sums nssq partials per token.
void fold_norm(GemmArgs& g, const dllm_model* m, const Workspace& w, int nssq) {
    g.ssq = w.ssq;
    g.nssq = nssq;
    g.ssq_ld = w.ssq_ld;
    g.dnorm = m->cfg.d_model;
    g.eps = m->cfg.eps;
}

template <int WT, typename AT>   // AT: element type of the embedding and the cache planes
int forward_t(dllm_model* m, dllm_kv* kv, const FwdArgs& a, hipStream_t s) {
    constexpr bool XF32 = (WT == WT_F32);
    const dllm_config& c = m->cfg;
    const int d = c.d_model, H = c.n_heads, Dh = c.head_dim;
    int rc = a.ws ? DLLM_OK : ensure_ws(m, a.M);
    if (rc) return rc;
    Workspace& w = a.ws ? *a.ws : m->ws;

    int MT, gy;
    if (a.M <= 64) { MT = pick_MT(a.M); gy = 1; }
    else { MT = 4; gy = ceil_div(a.M, 64); }
    const int Mc = gy * MT * 16;    // rows computed (padded)
    // Every kernel below touches token rows [0, Mc) of the workspace buffers.
    {
        const size_t need_d = (size_t)(Mc / 16) * m->KCx_d * XChunk<XF32>::bytes;
        const size_t need_f = (size_t)(Mc / 16) * m->KCx_f * XChunk<XF32>::bytes;
        if (Mc > w.rows || need_d > w.xg_bytes || need_d > w.of_bytes || need_f > w.af_bytes)
            return fail(DLLM_E_INVAL, "internal: workspace smaller than the launch extent");
        if (a.lm && Mc > w.wrows) return fail(DLLM_E_INVAL, "LM head rows exceed the window workspace");
    }

    // Windows of <= 64 rows fold each RMSNorm into the GEMM that consumes it: the
    // residual projections update x in their epilogue and leave x * g and per-tile
    // sums of squares; QKV, gate/up and the LM head scale their outputs per token.
    // Before a selective LM head (rows packed by need) the last layer writes the final
    // operand at each kept row's slot, which the embedding kernel records.
    const bool fused = (gy == 1);
    // The down projection keeps split-K + the reduction kernel (which writes the
    // normalised operand): over the whole K range each of its workgroups would read the
    // whole 12288-wide activation (4x the L2 traffic of 4 split-K slices).  QKV then
    // reads a normalised operand, except after the embedding (layer 0), which folds.
    constexpr bool FUSE_DOWN = false;
    const bool lm_sel_last = a.lm && a.sel;
    auto nssq_qkv = [&](int l) { return l == 0 ? 1 : m->layers[l - 1].down.n_tiles; };

    // replay (timing): the kernels of one class only, with the operands the workspace
    // holds, cycling through the layers
    auto run = [&](int cls) { return a.replay < 0 || a.replay == cls; };
    if (a.replay < 0)
        hipLaunchKernelGGL((embed_kernel<AT, XF32>), dim3(Mc), dim3(ROW_NT), 0, s, (const AT*)m->embed, a.tok,
                           a.mask, a.M, d, c.vocab, c.mask_id, c.eps, (const float*)m->layers[0].g1, w.x, w.xg,
                           m->KCx_d, fused ? w.ssq : nullptr, w.ssq_ld, (fused && lm_sel_last) ? w.slot : nullptr, a.need,
                           a.n_sel);

    // Cache per layer: [K][V^T], fp32 or fp16; Hkv heads.  Q: fp32, or fp16 hi / lo planes.
    const size_t plane = (size_t)m->Hkv * kv->Cs * Dh;
    const size_t layer_elems = 2 * plane;
    const size_t q_plane = XF32 ? 0 : (size_t)w.rows * d;
    const int n_iter = a.replay < 0 ? a.n_layers : (a.replay == DLLM_K_LMHEAD ? 0 : a.n_replay);
    for (int it = 0; it < n_iter; ++it) {
        const int l = it % c.n_layers;
        LayerW& L = m->layers[l];
        AT* Kc = (AT*)kv->buf + (size_t)l * layer_elems;
        AT* Vt = Kc + plane;

        // RMSNorm + QKV + RoPE -> Q buffer and K/V cache rows
        if (run(DLLM_K_QKV)) {
            GemmArgs g{L.qkv.w, L.qkv.scale, w.xg, L.qkv.KCw, L.qkv.KCw * WTraits<WT>::XPER, L.qkv.n_tiles, L.bqkv};
            g.qs = L.qkv.qs;
            if (fused && (l == 0 || FUSE_DOWN)) fold_norm(g, m, w, nssq_qkv(l));
            EpiQKV<XF32> e{d, m->dkv, Dh, a.M, a.pos_base, a.pos, m->rope, (AT*)w.q, q_plane, Kc, Vt, kv->Cs};
            ProbeScope ps(m, DLLM_K_QKV, s);
            if ((rc = launch_gemm<WT, G_QKV>(decomp(G_QKV, WT, L.qkv.n_tiles, Mc, gy), L.qkv.n_tiles, MT, g, e, gy, s,
                                             w.part, w.part_floats)))
                return rc;
        }
        // attention over [0, T) (+ split merge)
        if (run(DLLM_K_ATTN)) {
            AttnArgs at{};
            at.q = w.q; at.q_plane = q_plane; at.K = Kc; at.Vt = Vt; at.Cs = kv->Cs; at.H = H;
            at.G = H / m->Hkv; at.T = a.T; at.lim = a.lim; at.M = a.M;
            at.scale = 1.0f / sqrtf((float)Dh); at.o = w.of; at.KCx = m->KCx_d;
            at.opart = w.opart; at.mlpart = w.mlpart; at.rows_ld = w.wrows;
            ProbeScope ps(m, DLLM_K_ATTN, s);
            if (XF32) {
                at.nsplit = 1; at.bps = 1 << 20;
                if (Dh == 32) hipLaunchKernelGGL((attn_f32_kernel<32>), dim3(Mc, H), dim3(64), 0, s, at);
                else if (Dh == 64) hipLaunchKernelGGL((attn_f32_kernel<64>), dim3(Mc, H), dim3(64), 0, s, at);
                else hipLaunchKernelGGL((attn_f32_kernel<128>), dim3(Mc, H), dim3(64), 0, s, at);
            } else if (gy == 1 && Mc >= 48 && ceil_div(a.T, 32) <= ATTN_KEYGROUP_BLOCKS) {
                // windows of 48-64 rows over up to 1536 keys: the workgroup's QG query tiles
                // share each staged block and KS = 2 key groups take alternate blocks
                // (8 waves stage 2 blocks at a time); key splits across workgroups where a
                // group would take more than ATTN_ROUNDS blocks.  LLaDA-8B, 64 rows,
                // prefix 1024: 17.5 against 20.0 us per layer for one key group.  For 32
                // rows, and for long prefixes, one group per workgroup and the most splits
                // are faster (prefix 512: 13.3 against 14.9-15.8 us; 4096: 32.4 against 34.1).
                const int QGs = Mc / 16;                   // 3 or 4
                const int KSs = 2;
                const int nblk = ceil_div(a.T, 32);
                int nsplit = std::min(ceil_div(nblk, KSs * ATTN_ROUNDS), MAX_SPLIT);
                at.bps = ceil_div(nblk, nsplit);
                at.nsplit = ceil_div(nblk, at.bps);
                dim3 grid(at.nsplit * H);
#define ATTN_W(DH_, QG_, KS_) hipLaunchKernelGGL((attn_f16_kernel<DH_, QG_, KS_, 2>), grid, dim3(QG_ * KS_ * 64), 0, s, at)
#define ATTN_W_QG(DH_) \
    do { if (QGs == 3) ATTN_W(DH_, 3, 2); else ATTN_W(DH_, 4, 2); } while (0)
                if (Dh == 128) ATTN_W_QG(128); else ATTN_W_QG(64);
#undef ATTN_W_QG
#undef ATTN_W
                if (at.nsplit > 1)
                    hipLaunchKernelGGL((attn_combine_kernel<false>), dim3(ceil_div(Mc * H, ATTN_MERGE_PAIRS)),
                                       dim3(32 * ATTN_MERGE_PAIRS), 0, s, at,
                                       Mc, Dh);
            } else {
                // QG query tiles share each staged K/V block; key splits across
                // workgroups give the chip enough waves (~2 per SIMD) and are merged
                // by attn_combine
                // long prompts: 8 query tiles per workgroup halve the K/V blocks staged per
                // query (4096 tokens, 32 heads: 984 against 1149 us per layer) once that
                // still leaves 512+ workgroups
                const int QG = (a.M > 64 && Mc % 128 == 0 && (long)H * (Mc / 128) >= 512) ? 8
                               : (Mc >= 64) ? 4 : Mc / 16;
                const int nqg = Mc / (16 * QG);
                const int nblk = ceil_div(a.T, 32);
                int nsplit = std::max(1, std::min(nblk, 2048 / (H * nqg * QG)));
                if (a.M > 64) nsplit = std::min(nsplit, 1);          // prefill: enough workgroups already
                nsplit = std::min(nsplit, MAX_SPLIT);
                // at least 3 blocks per split: fewer partials to merge where the prefix is
                // short (LLaDA-8B, 32 rows, prefix 512: 6 splits of 3 blocks against 9 of 2,
                // attention + merge 11.0 -> 10.5 us; 4 blocks: 11.0)
                at.bps = std::max(ceil_div(nblk, nsplit), 3);
                at.nsplit = ceil_div(nblk, at.bps);
                dim3 grid(at.nsplit * H * nqg);
#define ATTN(DH_, QG_) hipLaunchKernelGGL((attn_f16_kernel<DH_, QG_, 1, ATTN_RING>), grid, dim3(QG_ * 64), 0, s, at)
#define ATTN_QG(DH_) \
    do { if (QG == 8) ATTN(DH_, 8); else if (QG == 4) ATTN(DH_, 4); else if (QG == 3) ATTN(DH_, 3); \
         else if (QG == 2) ATTN(DH_, 2); \
         else ATTN(DH_, 1); } while (0)
                if (Dh == 128) ATTN_QG(128); else ATTN_QG(64);
#undef ATTN_QG
#undef ATTN
                if (at.nsplit > 1) {
                    hipLaunchKernelGGL((attn_combine_kernel<false>), dim3(ceil_div(Mc * H, ATTN_MERGE_PAIRS)),
                                       dim3(32 * ATTN_MERGE_PAIRS), 0, s, at,
                                       Mc, Dh);
                }
            }
        }
        // O projection + residual (+ the norm-2 operand)
        if (run(DLLM_K_OPROJ)) {
            ProbeScope ps(m, DLLM_K_OPROJ, s);
            if (fused) {
                if ((rc = residual_proj_fused<WT, XF32>(m, w, L.o, w.of, L.g2, a.M, MT, s))) return rc;
            } else if ((rc = residual_proj<WT, XF32>(m, w, L.o, w.of, L.g2, a.M, Mc, MT, gy, s))) {
                return rc;
            }
        }
        // RMSNorm + gate/up + SwiGLU
        if (run(DLLM_K_GATEUP)) {
            GemmArgs g{L.gu.w, L.gu.scale, w.xg, L.gu.KCw, L.gu.KCw * WTraits<WT>::XPER, L.gu.n_tiles};
            g.qs = L.gu.qs;
            if (fused) fold_norm(g, m, w, L.o.n_tiles);
            EpiSwiGLU<XF32> e{w.af, m->KCx_f};
            ProbeScope ps(m, DLLM_K_GATEUP, s);
            if ((rc = launch_gemm<WT, G_GU>(decomp(G_GU, WT, L.gu.n_tiles, Mc, gy), L.gu.n_tiles, MT, g, e, gy, s)))
                return rc;
        }
        // down projection + residual (+ next norm operand)
        if (run(DLLM_K_DOWN)) {
            const bool last = (l + 1 == c.n_layers);
            const float* gnext = last ? m->gf : m->layers[l + 1].g1;
            const bool sel = last && lm_sel_last;
            ProbeScope ps(m, DLLM_K_DOWN, s);
            if (fused && FUSE_DOWN) {
                if ((rc = residual_proj_fused<WT, XF32>(m, w, L.down, w.af, gnext, a.M, MT, s, sel ? w.slot : nullptr)))
                    return rc;
            } else if ((rc = residual_proj<WT, XF32>(m, w, L.down, w.af, gnext, a.M, Mc, MT, gy, s, sel, a.need,
                                                     a.n_sel))) {
                return rc;
            }
        }
    }
    if (a.xout) HIP_TRY(hipMemcpyAsync(a.xout, w.x, (size_t)a.M * d * 4, hipMemcpyDeviceToDevice, s));
    if (a.lm || a.replay == DLLM_K_LMHEAD) {
        // rows the LM head runs over: all M, or the selected ones packed to the front
        const int Ml = a.sel ? std::min(a.n_sel, a.M) : a.M;
        int MTl = MT, gyl = gy;
        if (a.sel) {
            if (Ml <= 64) { MTl = pick_MT(std::max(Ml, 1)); gyl = 1; }
            else { MTl = 4; gyl = ceil_div(Ml, 64); }
        }
        if (gyl * MTl * 16 > w.wrows) return fail(DLLM_E_INVAL, "LM head rows exceed the window workspace");
        GemmArgs g{m->lm.w, m->lm.scale, w.xg, m->lm.KCw, m->lm.KCw * WTraits<WT>::XPER, m->lm.n_tiles};
        g.qs = m->lm.qs;
        if (fused && FUSE_DOWN) fold_norm(g, m, w, m->layers[c.n_layers - 1].down.n_tiles);
        const Decomp dc = decomp(G_LM, WT, m->lm.n_tiles, gyl * MTl * 16, gyl);
        const int gx = row_groups(dc, m->lm.n_tiles);
        if (gx > m->n_lm_wg) return fail(DLLM_E_INVAL, "internal: LM-head partials exceed their buffer");
        if (Ml > 0) {
            EpiLM e{c.vocab, c.mask_id, Ml, w.lm, w.wrows, a.logits};
            for (int r = 0; r < (a.replay < 0 ? 1 : a.n_replay); ++r) {
                ProbeScope ps(m, DLLM_K_LMHEAD, s);
                if ((rc = launch_gemm<WT, G_LM>(dc, m->lm.n_tiles, MTl, g, e, gyl, s))) return rc;
            }
        }
        if (a.replay < 0)
            hipLaunchKernelGGL(lm_combine_kernel, dim3(a.M), dim3(64), 0, s, (const LmPartial*)w.lm, gx, w.wrows,
                               a.out_id, a.out_conf, a.sel, a.need, a.n_sel, a.M);
    }
    HIP_TRY(hipGetLastError());
    return DLLM_OK;
}

int forward(dllm_model* m, dllm_kv* kv, const FwdArgs& a, hipStream_t s) {
    if (m->wt == WT_F32) return forward_t<WT_F32, float>(m, kv, a, s);
    if (m->wt == WT_BF16) return forward_t<WT_BF16, uint16_t>(m, kv, a, s);
    if (m->wt == WT_Q4) return forward_t<WT_Q4, uint16_t>(m, kv, a, s);
    return forward_t<WT_I8, uint16_t>(m, kv, a, s);
}

int check_model_kv(const dllm_model* m, const dllm_kv* kv) {
    if (!m) return fail(DLLM_E_INVAL, "model is NULL");
    if (!kv) return fail(DLLM_E_INVAL, "kv is NULL");
    if (kv->model != m) return fail(DLLM_E_INVAL, "kv cache belongs to another model");
    return DLLM_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
// Static scratch of the no-allocation step (dllm_denoise_step_noalloc): the step's
// workspaces carved from this array instead of the model's.  Each device holds its
// own copy (at its own address) until the process ends.  Host code never passes
// the array's name to a kernel: it resolves the device address once per device with
// hipGetSymbolAddress and uses that pointer.
// ---------------------------------------------------------------------------
static constexpr size_t SCRATCH_BYTES = (size_t)64 << 20;
static __device__ __align__(256) char scratch[SCRATCH_BYTES];

namespace {

constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[MAX_DEVICES] = {};

// Device address of `scratch` on the current device (resolved on the first call per device).
int scratch_ptr(void** out) {
    int dev = -1;
    HIP_TRY(hipGetDevice(&dev));
    if (dev < 0 || dev >= MAX_DEVICES) return fail(DLLM_E_INVAL, "device index out of range for the static scratch");
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        if (!p) return fail(DLLM_E_HIP, "hipGetSymbolAddress returned NULL for the static scratch");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return DLLM_OK;
}

}  // namespace

// ===========================================================================
// C ABI
// ===========================================================================

extern "C" {

const char* dllm_last_error(void) { return g_last_error.c_str(); }

const char* dllm_version(void) { return "dllm-gfx950 0.1"; }

int dllm_model_create(const dllm_config* cfg, const dllm_weights* w, dllm_stream stream, dllm_model** out) {
    if (!out) return fail(DLLM_E_INVAL, "out is NULL");
    *out = nullptr;
    int rc = validate_config(cfg);
    if (rc) return rc;
    if (!w || !w->embed || !w->lm_head || !w->final_norm || !w->layers)
        return fail(DLLM_E_INVAL, "weights: NULL pointer");
    for (int l = 0; l < cfg->n_layers; ++l) {
        const dllm_layer_weights& L = w->layers[l];
        if (!L.wq || !L.wk || !L.wv || !L.wo || !L.wg || !L.wu || !L.wd || !L.attn_norm || !L.ffn_norm)
            return fail(DLLM_E_INVAL, "weights: NULL pointer in layer " + std::to_string(l));
        if (cfg->qkv_bias && (!L.bq || !L.bk || !L.bv))
            return fail(DLLM_E_INVAL, "weights: NULL bias pointer in layer " + std::to_string(l));
    }
    hipStream_t s = (hipStream_t)stream;
    dllm_model* m = new dllm_model();
    m->cfg = *cfg;
    const dllm_config& c = m->cfg;
    m->wt = c.dtype == DLLM_F32 ? WT_F32 : (c.dtype == DLLM_BF16 ? WT_BF16 : (c.dtype == DLLM_W8 ? WT_I8 : WT_Q4));
    m->xf32 = c.dtype == DLLM_F32;
    m->kv_elem = m->xf32 ? 4 : 2;
    m->Hkv = c.n_kv_heads > 0 ? c.n_kv_heads : c.n_heads;
    m->dkv = m->Hkv * c.head_dim;
    const int xcols = m->xf32 ? 16 : 32;
    const int xper = (m->wt == WT_I8 || m->wt == WT_Q4) ? 2 : 1;
    const int d = c.d_model, F = c.d_ff;

    m->layers.resize(c.n_layers);
    size_t wbytes = 0, srows = 0, qbytes = 0;
    for (auto& L : m->layers) {
        plan_packed(L.qkv, m->wt, d + 2 * m->dkv, d);
        plan_packed(L.o, m->wt, d, d);
        plan_packed(L.gu, m->wt, 2 * F, d);
        plan_packed(L.down, m->wt, d, F);
        for (PackedW* p : {&L.qkv, &L.o, &L.gu, &L.down}) {
            wbytes += p->bytes;
            srows += p->n_tiles * 16;
            qbytes += p->qs_bytes;
        }
    }
    plan_packed(m->lm, m->wt, c.vocab, d);
    wbytes += m->lm.bytes;
    srows += m->lm.n_tiles * 16;
    qbytes += m->lm.qs_bytes;
    m->KCx_d = m->layers[0].qkv.KCw * xper;
    m->KCx_f = m->layers[0].down.KCw * xper;
    (void)xcols;
    m->n_lm_wg = m->lm.n_tiles;   // row groups of any LM-head launch (at least one tile each)

    auto cleanup = [&](int code) {
        dllm_model_destroy(m);
        return code;
    };
    if ((rc = alloc_zero(&m->wpool, wbytes))) return cleanup(rc);
    if (m->wt == WT_I8 && (rc = alloc_zero((void**)&m->spool, srows * 4))) return cleanup(rc);
    if (m->wt == WT_Q4 && (rc = alloc_zero((void**)&m->qpool, qbytes))) return cleanup(rc);
    if ((rc = alloc_zero((void**)&m->gpool, (size_t)(2 * c.n_layers + 1) * d * 4))) return cleanup(rc);
    const int qkv_rows = m->layers[0].qkv.n_tiles * 16;     // packed (padded) Q/K/V rows
    if (c.qkv_bias && (rc = alloc_zero((void**)&m->bpool, (size_t)c.n_layers * qkv_rows * 4))) return cleanup(rc);
    const size_t esize = m->xf32 ? 4 : 2;
    if ((rc = alloc_zero(&m->embed, (size_t)c.vocab * d * esize))) return cleanup(rc);
    const int half = c.head_dim / 2;
    if ((rc = alloc_zero((void**)&m->rope, (size_t)c.max_pos * half * sizeof(float2)))) return cleanup(rc);

    // carve
    char* wp = (char*)m->wpool;
    float* sp = m->spool;
    char* qp = (char*)m->qpool;
    auto carve = [&](PackedW& p) {
        p.w = wp;
        wp += p.bytes;
        if (sp) { p.scale = sp; sp += p.n_tiles * 16; }
        if (qp) { p.qs = (uint16_t*)qp; qp += p.qs_bytes; }
    };
    for (auto& L : m->layers) { carve(L.qkv); carve(L.o); carve(L.gu); carve(L.down); }
    carve(m->lm);
    for (int l = 0; l < c.n_layers; ++l) {
        m->layers[l].g1 = m->gpool + (size_t)(2 * l) * d;
        m->layers[l].g2 = m->gpool + (size_t)(2 * l + 1) * d;
        if (m->bpool) m->layers[l].bqkv = m->bpool + (size_t)l * qkv_rows;
    }
    m->gf = m->gpool + (size_t)(2 * c.n_layers) * d;

    // pack
    const bool src_f32 = (c.dtype == DLLM_F32);
    auto pack = [&](PackedW& p, int kind, const void* a0, const void* a1, const void* a2) -> int {
        PackSrc src{{a0, a1, a2}, kind, p.N, p.K, d, c.head_dim, m->dkv};
        return src_f32 ? pack_one<float>(m, p, src, s) : pack_one<uint16_t>(m, p, src, s);
    };
    for (int l = 0; l < c.n_layers; ++l) {
        const dllm_layer_weights& S = w->layers[l];
        LayerW& L = m->layers[l];
        if ((rc = pack(L.qkv, MAP_QKV, S.wq, S.wk, S.wv))) return cleanup(rc);
        if (L.bqkv) {
            PackSrc bs{{S.bq, S.bk, S.bv}, MAP_QKV, L.qkv.N, 1, d, c.head_dim, m->dkv};
            hipLaunchKernelGGL(pack_bias_kernel, dim3(ceil_div(qkv_rows, 256)), dim3(256), 0, s, bs, qkv_rows, L.bqkv);
        }
        if ((rc = pack(L.o, MAP_IDENT, S.wo, nullptr, nullptr))) return cleanup(rc);
        if ((rc = pack(L.gu, MAP_GATEUP, S.wg, S.wu, nullptr))) return cleanup(rc);
        if ((rc = pack(L.down, MAP_IDENT, S.wd, nullptr, nullptr))) return cleanup(rc);
        if (hipMemcpyAsync(L.g1, S.attn_norm, d * 4, hipMemcpyDeviceToDevice, s) != hipSuccess ||
            hipMemcpyAsync(L.g2, S.ffn_norm, d * 4, hipMemcpyDeviceToDevice, s) != hipSuccess)
            return cleanup(fail(DLLM_E_HIP, "copying norm gains failed"));
    }
    if ((rc = pack(m->lm, MAP_IDENT, w->lm_head, nullptr, nullptr))) return cleanup(rc);
    if (hipMemcpyAsync(m->gf, w->final_norm, d * 4, hipMemcpyDeviceToDevice, s) != hipSuccess ||
        hipMemcpyAsync(m->embed, w->embed, (size_t)c.vocab * d * esize, hipMemcpyDeviceToDevice, s) != hipSuccess)
        return cleanup(fail(DLLM_E_HIP, "copying embedding / final norm failed"));
    {
        const size_t n = (size_t)c.max_pos * half;
        hipLaunchKernelGGL(rope_table_kernel, dim3(ceil_div((long)n, 256)), dim3(256), 0, s, m->rope, c.max_pos, half,
                           (double)c.rope_base);
    }
    if (hipGetLastError() != hipSuccess || hipStreamSynchronize(s) != hipSuccess)
        return cleanup(fail(DLLM_E_HIP, "weight prepacking failed"));
    if ((rc = ensure_ws(m, c.max_window))) return cleanup(rc);
    {
        void* sp = nullptr;     // resolve the static scratch of this device while it is current
        if ((rc = scratch_ptr(&sp))) return cleanup(rc);
    }
    *out = m;
    return DLLM_OK;
}

int dllm_model_destroy(dllm_model* m) {
    if (!m) return DLLM_OK;
    free_ws(m->ws);
    void* ptrs[] = {m->wpool, m->spool, m->qpool, m->gpool, m->bpool, m->embed, m->rope};
    for (void* p : ptrs)
        if (p) (void)hipFree(p);
    for (auto e : m->ev_b) (void)hipEventDestroy(e);
    for (auto e : m->ev_e) (void)hipEventDestroy(e);
    delete m;
    return DLLM_OK;
}

static int cs_of(int capacity) { return (int)round_up(capacity, 32); }

int dllm_kv_bytes(const dllm_model* m, int32_t capacity, size_t* bytes) {
    if (!m || !bytes) return fail(DLLM_E_INVAL, "NULL argument");
    if (capacity < 1 || capacity > m->cfg.max_pos)
        return fail(DLLM_E_CAPACITY, "capacity must be in [1, max_pos]");
    const dllm_config& c = m->cfg;
    *bytes = (size_t)c.n_layers * 2 * m->Hkv * cs_of(capacity) * c.head_dim * m->kv_elem;
    return DLLM_OK;
}

int dllm_kv_create(const dllm_model* m, void* d_buf, size_t bytes, int32_t capacity, dllm_kv** out) {
    if (!out) return fail(DLLM_E_INVAL, "out is NULL");
    *out = nullptr;
    size_t need = 0;
    int rc = dllm_kv_bytes(m, capacity, &need);
    if (rc) return rc;
    if (!d_buf) return fail(DLLM_E_INVAL, "buffer is NULL");
    if (bytes < need) return fail(DLLM_E_CAPACITY, "buffer smaller than dllm_kv_bytes()");
    if (((uintptr_t)d_buf & 15) != 0) return fail(DLLM_E_INVAL, "buffer must be 16-byte aligned");
    *out = new dllm_kv{m, d_buf, bytes, capacity, cs_of(capacity), 0, 0};
    return DLLM_OK;
}

int dllm_kv_destroy(dllm_kv* kv) {
    delete kv;
    return DLLM_OK;
}

int dllm_kv_prefix_len(const dllm_kv* kv, int32_t* prefix_len, int32_t* prompt_len) {
    if (!kv) return fail(DLLM_E_INVAL, "kv is NULL");
    if (prefix_len) *prefix_len = kv->prefix_len;
    if (prompt_len) *prompt_len = kv->prompt_len;
    return DLLM_OK;
}

int dllm_kv_set_prefix_len(dllm_kv* kv, int32_t prefix_len) {
    if (!kv) return fail(DLLM_E_INVAL, "kv is NULL");
    if (prefix_len < kv->prompt_len || prefix_len > kv->capacity)
        return fail(DLLM_E_INVAL, "prefix_len must be in [prompt_len, capacity]");
    kv->prefix_len = prefix_len;
    return DLLM_OK;
}

int dllm_prefill(dllm_model* m, dllm_kv* kv, const int32_t* d_ids, int32_t n, dllm_stream stream) {
    int rc = check_model_kv(m, kv);
    if (rc) return rc;
    if (!d_ids) return fail(DLLM_E_INVAL, "ids is NULL");
    if (n < 1) return fail(DLLM_E_INVAL, "n must be >= 1");
    if (kv->prefix_len != 0) return fail(DLLM_E_INVAL, "prefill needs an empty cache");
    if (n > kv->capacity) return fail(DLLM_E_CAPACITY, "prompt longer than the cache capacity");
    FwdArgs a{};
    a.M = n; a.tok = d_ids; a.mask = nullptr; a.pos_base = 0; a.pos = nullptr; a.T = n; a.lim = nullptr;
    a.n_layers = m->cfg.n_layers; a.lm = false;
    if ((rc = forward(m, kv, a, (hipStream_t)stream))) return rc;
    kv->prefix_len = n;
    kv->prompt_len = n;
    return DLLM_OK;
}

static int window_checks(dllm_model* m, dllm_kv* kv, const int32_t* d_tok, int32_t W) {
    int rc = check_model_kv(m, kv);
    if (rc) return rc;
    if (!d_tok) return fail(DLLM_E_INVAL, "tokens pointer is NULL");
    if (W < 1 || W > m->cfg.max_window) return fail(DLLM_E_INVAL, "W must be in [1, max_window]");
    if (kv->prefix_len + W > kv->capacity) return fail(DLLM_E_CAPACITY, "prefix_len + W exceeds the cache capacity");
    return DLLM_OK;
}

int dllm_denoise_step(dllm_model* m, dllm_kv* kv, const int32_t* d_tok, const uint8_t* d_mask, int32_t W,
                      int32_t* d_out_id, float* d_out_conf, dllm_stream stream) {
    int rc = window_checks(m, kv, d_tok, W);
    if (rc) return rc;
    if (!d_out_id || !d_out_conf) return fail(DLLM_E_INVAL, "output pointer is NULL");
    FwdArgs a{};
    a.M = W; a.tok = d_tok; a.mask = d_mask; a.pos_base = kv->prefix_len; a.T = kv->prefix_len + W;
    a.n_layers = m->cfg.n_layers; a.lm = true; a.out_id = d_out_id; a.out_conf = d_out_conf;
    return forward(m, kv, a, (hipStream_t)stream);
}

int dllm_denoise_step_noalloc(dllm_model* m, dllm_kv* kv, const int32_t* d_tok, const uint8_t* d_mask, int32_t W,
                              int32_t* d_out_id, float* d_out_conf, dllm_stream stream) {
    int rc = window_checks(m, kv, d_tok, W);
    if (rc) return rc;
    if (!d_out_id || !d_out_conf) return fail(DLLM_E_INVAL, "output pointer is NULL");
    const int rows = (int)round_up(W, 64);
    const size_t part_floats = part_floats_for(m, rows, rows);
    const size_t need = ws_carve(m, rows, rows, part_floats, nullptr, nullptr);
    if (need > SCRATCH_BYTES)
        return fail(DLLM_E_CAPACITY, "the step needs " + std::to_string(need) + " bytes of scratch; the static scratch holds " +
                                         std::to_string(SCRATCH_BYTES));
    void* base = nullptr;
    if ((rc = scratch_ptr(&base))) return rc;
    Workspace w;
    ws_carve(m, rows, rows, part_floats, (char*)base, &w);
    // padding columns of the activation fragments (widths that are not whole chunks):
    // never written by the step, multiplied by zero weights, so they must be zeros
    const int kcol = m->xf32 ? 16 : 32;
    const struct { void* buf; int KCx, kreal; } pads[] = {
        {w.xg, m->KCx_d, m->cfg.d_model}, {w.of, m->KCx_d, m->cfg.d_model}, {w.af, m->KCx_f, m->cfg.d_ff}};
    for (const auto& pd : pads) {
        if (pd.KCx * kcol == pd.kreal) continue;
        const long n = (long)(rows / 16) * (pd.KCx - pd.kreal / kcol) * 64 * (m->xf32 ? 1 : 2);
        if (m->xf32)
            hipLaunchKernelGGL(zero_frag_pad_kernel<true>, dim3(ceil_div(n, 256)), dim3(256), 0, (hipStream_t)stream,
                               pd.buf, rows / 16, pd.KCx, pd.kreal);
        else
            hipLaunchKernelGGL(zero_frag_pad_kernel<false>, dim3(ceil_div(n, 256)), dim3(256), 0, (hipStream_t)stream,
                               pd.buf, rows / 16, pd.KCx, pd.kreal);
    }
    FwdArgs a{};
    a.M = W; a.tok = d_tok; a.mask = d_mask; a.pos_base = kv->prefix_len; a.T = kv->prefix_len + W;
    a.n_layers = m->cfg.n_layers; a.lm = true; a.out_id = d_out_id; a.out_conf = d_out_conf; a.ws = &w;
    return forward(m, kv, a, (hipStream_t)stream);
}

int dllm_denoise_window(dllm_model* m, dllm_kv* kv, int32_t w0, const int32_t* d_tok, const uint8_t* d_mask,
                        int32_t W, int32_t* d_out_id, float* d_out_conf, dllm_stream stream) {
    int rc = check_model_kv(m, kv);
    if (rc) return rc;
    if (!d_tok || !d_out_id || !d_out_conf) return fail(DLLM_E_INVAL, "NULL argument");
    if (W < 1 || W > m->cfg.max_window) return fail(DLLM_E_INVAL, "W must be in [1, max_window]");
    if (w0 < kv->prefix_len) return fail(DLLM_E_INVAL, "w0 must be >= prefix_len");
    if ((long)w0 + W > kv->capacity) return fail(DLLM_E_CAPACITY, "w0 + W exceeds the cache capacity");
    FwdArgs a{};
    a.M = W; a.tok = d_tok; a.mask = d_mask; a.pos_base = w0; a.T = w0 + W;
    a.n_layers = m->cfg.n_layers; a.lm = true; a.out_id = d_out_id; a.out_conf = d_out_conf;
    return forward(m, kv, a, (hipStream_t)stream);
}

int dllm_denoise_window_sls(dllm_model* m, dllm_kv* kv, int32_t w0, const int32_t* d_tok, const uint8_t* d_mask,
                            const uint8_t* d_need, int32_t n_need, int32_t W, int32_t* d_out_id, float* d_out_conf,
                            dllm_stream stream) {
    int rc = check_model_kv(m, kv);
    if (rc) return rc;
    if (!d_tok || !d_out_id || !d_out_conf) return fail(DLLM_E_INVAL, "NULL argument");
    if (W < 1 || W > m->cfg.max_window) return fail(DLLM_E_INVAL, "W must be in [1, max_window]");
    if (n_need < 0 || n_need > W) return fail(DLLM_E_INVAL, "n_need must be in [0, W]");
    if (w0 < kv->prefix_len) return fail(DLLM_E_INVAL, "w0 must be >= prefix_len");
    if ((long)w0 + W > kv->capacity) return fail(DLLM_E_CAPACITY, "w0 + W exceeds the cache capacity");
    FwdArgs a{};
    a.M = W; a.tok = d_tok; a.mask = d_mask; a.pos_base = w0; a.T = w0 + W;
    a.n_layers = m->cfg.n_layers; a.lm = true; a.out_id = d_out_id; a.out_conf = d_out_conf;
    a.sel = true; a.need = d_need; a.n_sel = n_need;
    return forward(m, kv, a, (hipStream_t)stream);
}

int dllm_debug_logits(dllm_model* m, dllm_kv* kv, const int32_t* d_tok, const uint8_t* d_mask, int32_t W,
                      float* d_logits, int32_t* d_out_id, float* d_out_conf, dllm_stream stream) {
    int rc = window_checks(m, kv, d_tok, W);
    if (rc) return rc;
    if (!d_logits) return fail(DLLM_E_INVAL, "logits pointer is NULL");
    FwdArgs a{};
    a.M = W; a.tok = d_tok; a.mask = d_mask; a.pos_base = kv->prefix_len; a.T = kv->prefix_len + W;
    a.n_layers = m->cfg.n_layers; a.lm = true; a.logits = d_logits; a.out_id = d_out_id; a.out_conf = d_out_conf;
    return forward(m, kv, a, (hipStream_t)stream);
}

int dllm_debug_hidden(dllm_model* m, dllm_kv* kv, const int32_t* d_tok, const uint8_t* d_mask, int32_t W,
                      int32_t n_layers, float* d_x, dllm_stream stream) {
    int rc = window_checks(m, kv, d_tok, W);
    if (rc) return rc;
    if (!d_x) return fail(DLLM_E_INVAL, "output pointer is NULL");
    if (n_layers < 0 || n_layers > m->cfg.n_layers) return fail(DLLM_E_INVAL, "n_layers out of range");
    FwdArgs a{};
    a.M = W; a.tok = d_tok; a.mask = d_mask; a.pos_base = kv->prefix_len; a.T = kv->prefix_len + W;
    a.n_layers = n_layers; a.lm = false; a.xout = d_x;
    return forward(m, kv, a, (hipStream_t)stream);
}

int dllm_commit(const float* d_conf, const int32_t* d_id, int32_t* d_tok, uint8_t* d_mask, int32_t seg_begin,
                int32_t seg_len, int32_t k, int32_t* d_committed_pos, int32_t* d_n_committed, dllm_stream stream) {
    if (!d_conf || !d_id || !d_tok || !d_mask) return fail(DLLM_E_INVAL, "NULL argument");
    if (k < 0) return fail(DLLM_E_INVAL, "k must be >= 0");
    if (seg_begin < 0 || seg_len < 0 || seg_len > 1024) return fail(DLLM_E_INVAL, "segment out of range");
    hipLaunchKernelGGL(commit_kernel, dim3(1), dim3(256), 0, (hipStream_t)stream, d_conf, d_id, d_tok, d_mask,
                       seg_begin, seg_len, k, d_committed_pos, d_n_committed);
    HIP_TRY(hipGetLastError());
    return DLLM_OK;
}

int dllm_append_prefix_kv(dllm_model* m, dllm_kv* kv, const int32_t* d_block_tok, int32_t n, dllm_stream stream) {
    int rc = window_checks(m, kv, d_block_tok, n);
    if (rc) return rc;
    FwdArgs a{};
    a.M = n; a.tok = d_block_tok; a.pos_base = kv->prefix_len; a.T = kv->prefix_len + n;
    a.n_layers = m->cfg.n_layers; a.lm = false;
    if ((rc = forward(m, kv, a, (hipStream_t)stream))) return rc;
    kv->prefix_len += n;
    return DLLM_OK;
}

int dllm_refresh_kv(dllm_model* m, dllm_kv* kv, const int32_t* d_pos, const int32_t* d_new_id, int32_t n,
                    int32_t* d_out_id, float* d_out_conf, dllm_stream stream) {
    int rc = check_model_kv(m, kv);
    if (rc) return rc;
    if (!d_pos || !d_new_id) return fail(DLLM_E_INVAL, "NULL argument");
    if (n < 1 || n > m->cfg.max_window) return fail(DLLM_E_INVAL, "n must be in [1, max_window]");
    if ((d_out_id == nullptr) != (d_out_conf == nullptr))
        return fail(DLLM_E_INVAL, "out_id and out_conf must both be set or both be NULL");
    hipStream_t s = (hipStream_t)stream;
    std::vector<int32_t> pos(n);
    HIP_TRY(hipMemcpyAsync(pos.data(), d_pos, (size_t)n * 4, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    std::vector<int32_t> sorted(pos);
    std::sort(sorted.begin(), sorted.end());
    for (int i = 0; i < n; ++i) {
        if (sorted[i] < 0 || sorted[i] >= kv->prefix_len)
            return fail(DLLM_E_INVAL, "refresh position outside [0, prefix_len)");
        if (i > 0 && sorted[i] == sorted[i - 1]) return fail(DLLM_E_INVAL, "refresh positions must be distinct");
    }
    int T = 0;
    for (int p : pos) {
        const int e = (p < kv->prompt_len) ? kv->prompt_len
                                           : kv->prompt_len + m->cfg.block * (1 + (p - kv->prompt_len) / m->cfg.block);
        T = std::max(T, std::min(e, kv->prefix_len));
    }
    if ((rc = ensure_ws(m, n))) return rc;
    HIP_TRY(hipMemcpyAsync(m->ws.pos, d_pos, (size_t)n * 4, hipMemcpyDeviceToDevice, s));
    hipLaunchKernelGGL(refresh_limits_kernel, dim3(ceil_div(n, 64)), dim3(64), 0, s, d_pos, n, kv->prompt_len,
                       m->cfg.block, kv->prefix_len, m->ws.lim);
    FwdArgs a{};
    a.M = n; a.tok = d_new_id; a.pos = m->ws.pos; a.T = T; a.lim = m->ws.lim;
    a.n_layers = m->cfg.n_layers; a.lm = d_out_id != nullptr; a.out_id = d_out_id; a.out_conf = d_out_conf;
    return forward(m, kv, a, s);
}

int dllm_step_merged(dllm_model* m, dllm_kv* kv, const int32_t* d_ref_pos, const int32_t* d_ref_id, int32_t n_ref,
                     const int32_t* d_block_tok, int32_t n_block, const int32_t* d_tok, const uint8_t* d_mask,
                     int32_t W, int32_t* d_out_id, float* d_out_conf, int32_t* d_ref_out_id, float* d_ref_out_conf,
                     dllm_stream stream) {
    int rc = check_model_kv(m, kv);
    if (rc) return rc;
    if (n_ref < 0 || n_block < 0 || W < 0) return fail(DLLM_E_INVAL, "row counts must be >= 0");
    const int M = n_ref + n_block + W;
    if (M < 1 || M > m->cfg.max_window) return fail(DLLM_E_INVAL, "n_ref + n_block + W must be in [1, max_window]");
    if ((n_ref > 0 && (!d_ref_pos || !d_ref_id)) || (n_block > 0 && !d_block_tok) || (W > 0 && !d_tok))
        return fail(DLLM_E_INVAL, "NULL input pointer for a non-empty row group");
    if ((d_out_id == nullptr) != (d_out_conf == nullptr) || (d_ref_out_id == nullptr) != (d_ref_out_conf == nullptr))
        return fail(DLLM_E_INVAL, "each id / conf output pair must be both set or both NULL");
    const int P = kv->prefix_len;
    if (P + n_block + W > kv->capacity) return fail(DLLM_E_CAPACITY, "prefix_len + n_block + W exceeds the capacity");
    hipStream_t s = (hipStream_t)stream;
    if (n_ref > 0) {
        std::vector<int32_t> pos(n_ref);
        HIP_TRY(hipMemcpyAsync(pos.data(), d_ref_pos, (size_t)n_ref * 4, hipMemcpyDeviceToHost, s));
        HIP_TRY(hipStreamSynchronize(s));
        std::sort(pos.begin(), pos.end());
        for (int i = 0; i < n_ref; ++i) {
            if (pos[i] < 0 || pos[i] >= P) return fail(DLLM_E_INVAL, "refresh position outside [0, prefix_len)");
            if (i > 0 && pos[i] == pos[i - 1]) return fail(DLLM_E_INVAL, "refresh positions must be distinct");
        }
    }
    if ((rc = ensure_ws(m, M))) return rc;
    Workspace& w = m->ws;
    // the LM head runs only over the rows whose outputs are asked for (the appended
    // block's rows never need one)
    const bool ref_out = d_ref_out_id != nullptr && n_ref > 0, win_out = d_out_id != nullptr && W > 0;
    hipLaunchKernelGGL(merged_rows_kernel, dim3(ceil_div(M, 64)), dim3(64), 0, s, d_ref_pos, d_ref_id, n_ref,
                       d_block_tok, n_block, d_tok, d_mask, W, P, kv->prompt_len, m->cfg.block, (int)ref_out,
                       (int)win_out, w.tok, w.msk, w.pos, w.lim, w.need);
    const bool lm = ref_out || win_out;
    const int n_sel = (ref_out ? n_ref : 0) + (win_out ? W : 0);
    FwdArgs a{};
    a.M = M; a.tok = w.tok; a.mask = w.msk; a.pos = w.pos; a.T = P + n_block + W; a.lim = w.lim;
    a.n_layers = m->cfg.n_layers; a.lm = lm; a.out_id = w.oid; a.out_conf = w.oconf;
    a.sel = n_sel < M; a.need = w.need; a.n_sel = n_sel;
    if ((rc = forward(m, kv, a, s))) return rc;
    if (lm) {
        hipLaunchKernelGGL(merged_out_kernel, dim3(ceil_div(M, 64)), dim3(64), 0, s, (const int*)w.oid,
                           (const float*)w.oconf, n_ref, n_block, W, d_ref_out_id, d_ref_out_conf, d_out_id, d_out_conf);
        HIP_TRY(hipGetLastError());
    }
    kv->prefix_len = P + n_block;
    return DLLM_OK;
}

int dllm_probe_enable(dllm_model* m, int32_t kernel_class, int32_t max_records) {
    if (!m) return fail(DLLM_E_INVAL, "model is NULL");
    if (kernel_class < 0) { m->probe_class = -1; return DLLM_OK; }
    if (kernel_class > DLLM_K_LMHEAD || max_records < 1) return fail(DLLM_E_INVAL, "bad probe arguments");
    while ((int)m->ev_b.size() < max_records) {
        hipEvent_t b, e;
        HIP_TRY(hipEventCreate(&b));
        HIP_TRY(hipEventCreate(&e));
        m->ev_b.push_back(b);
        m->ev_e.push_back(e);
    }
    m->probe_class = kernel_class;
    m->probe_max = max_records;
    m->probe_n = 0;
    return DLLM_OK;
}

int dllm_probe_read(dllm_model* m, int32_t* n_records, double* mean_ms) {
    if (!m || !n_records || !mean_ms) return fail(DLLM_E_INVAL, "NULL argument");
    double tot = 0;
    for (int i = 0; i < m->probe_n; ++i) {
        HIP_TRY(hipEventSynchronize(m->ev_e[i]));
        float ms = 0.f;
        HIP_TRY(hipEventElapsedTime(&ms, m->ev_b[i], m->ev_e[i]));
        tot += ms;
    }
    *n_records = m->probe_n;
    *mean_ms = m->probe_n ? tot / m->probe_n : 0.0;
    m->probe_n = 0;
    return DLLM_OK;
}

int dllm_kernel_replay(dllm_model* m, dllm_kv* kv, int32_t kernel_class, int32_t W, int32_t n_launches,
                       dllm_stream stream) {
    int rc = check_model_kv(m, kv);
    if (rc) return rc;
    if (kernel_class < 0 || kernel_class > DLLM_K_LMHEAD) return fail(DLLM_E_INVAL, "unknown kernel class");
    if (W < 1 || W > m->cfg.max_window) return fail(DLLM_E_INVAL, "W must be in [1, max_window]");
    if (n_launches < 1) return fail(DLLM_E_INVAL, "n_launches must be >= 1");
    if (kv->prefix_len + W > kv->capacity) return fail(DLLM_E_CAPACITY, "prefix_len + W exceeds the capacity");
    FwdArgs a{};
    a.M = W; a.tok = nullptr; a.mask = nullptr; a.pos_base = kv->prefix_len; a.T = kv->prefix_len + W;
    a.n_layers = m->cfg.n_layers; a.lm = false; a.replay = kernel_class; a.n_replay = n_launches;
    return forward(m, kv, a, (hipStream_t)stream);
}

int dllm_kernel_bytes(const dllm_model* m, int32_t kernel_class, int32_t W, int32_t P, double* bytes) {
    if (!m || !bytes) return fail(DLLM_E_INVAL, "NULL argument");
    const dllm_config& c = m->cfg;
    // What the method must move (no logits, no activations: those stay in L2): every
    // weight once (Q4_0: a 4-bit code plus a 2-byte scale per 32 weights; int8: plus a
    // 4-byte scale per row; Q/K/V biases), the K/V it reads and the K/V rows it writes
    // at one value per element (4 bytes for fp32 models, 2 otherwise).
    const double wsz = m->wt == WT_F32 ? 4.0 : (m->wt == WT_BF16 ? 2.0 : (m->wt == WT_I8 ? 1.0 : 0.5 + 2.0 / 32));
    const double vsz = m->wt == WT_F32 ? 4.0 : 2.0;
    const double d = c.d_model, F = c.d_ff, V = c.vocab, dkv = m->dkv;
    const double scale_b = (m->wt == WT_I8) ? 4.0 : 0.0;   // per weight row
    const double bias_b = c.qkv_bias ? 4.0 : 0.0;           // per Q/K/V row
    double b = 0;
    switch (kernel_class) {
        case DLLM_K_QKV: b = (d + 2 * dkv) * (d * wsz + scale_b + bias_b) + 2.0 * W * dkv * vsz; break;
        case DLLM_K_ATTN: b = 2.0 * (P + W) * dkv * vsz; break;
        case DLLM_K_OPROJ: b = d * d * wsz + d * scale_b; break;
        case DLLM_K_GATEUP: b = 2 * F * d * wsz + 2 * F * scale_b; break;
        case DLLM_K_DOWN: b = d * F * wsz + d * scale_b; break;
        case DLLM_K_LMHEAD: b = V * d * wsz + V * scale_b; break;
        default: return fail(DLLM_E_INVAL, "unknown kernel class");
    }
    *bytes = b;
    return DLLM_OK;
}

int dllm_commit_staged(const float* d_conf, const int32_t* d_id, int32_t* d_tok, uint8_t* d_mask,
                       uint8_t* d_state, int32_t seg_begin, int32_t seg_len, float theta_visible,
                       float theta_stable, int32_t* d_promoted_pos, int32_t* d_n_promoted, dllm_stream stream) {
    if (!d_conf || !d_id || !d_tok || !d_mask || !d_state) return fail(DLLM_E_INVAL, "NULL argument");
    if (seg_begin < 0 || seg_len < 1 || seg_len > 1024) return fail(DLLM_E_INVAL, "segment must hold 1..1024 rows");
    if (!std::isfinite(theta_visible) || !std::isfinite(theta_stable))
        return fail(DLLM_E_INVAL, "thresholds must be finite");
    hipLaunchKernelGGL(commit_staged_kernel, dim3(1), dim3(1024), 0, (hipStream_t)stream, d_conf, (const int*)d_id,
                       (int*)d_tok, d_mask, d_state, seg_begin, seg_len, theta_visible, theta_stable,
                       (int*)d_promoted_pos, (int*)d_n_promoted);
    HIP_TRY(hipGetLastError());
    return DLLM_OK;
}

int dllm_accept_drafts(const float* d_conf, const int32_t* d_id, const int32_t* d_draft_id, int32_t* d_tok,
                       uint8_t* d_mask, int32_t n, float theta, int32_t* d_accepted_pos, int32_t* d_n_accepted,
                       dllm_stream stream) {
    if (!d_conf || !d_id || !d_draft_id || !d_tok || !d_mask) return fail(DLLM_E_INVAL, "NULL argument");
    if (n < 1 || n > 1024) return fail(DLLM_E_INVAL, "n must be in [1, 1024]");
    if (!std::isfinite(theta)) return fail(DLLM_E_INVAL, "theta must be finite");
    hipLaunchKernelGGL(accept_drafts_kernel, dim3(1), dim3(1024), 0, (hipStream_t)stream, d_conf, (const int*)d_id,
                       (const int*)d_draft_id, (int*)d_tok, d_mask, n, theta, (int*)d_accepted_pos,
                       (int*)d_n_accepted);
    HIP_TRY(hipGetLastError());
    return DLLM_OK;
}

int dllm_record_drafts(const int32_t* d_id, const uint8_t* d_mask, int32_t* d_draft_id, int32_t n,
                       dllm_stream stream) {
    if (!d_id || !d_mask || !d_draft_id) return fail(DLLM_E_INVAL, "NULL argument");
    if (n < 1) return fail(DLLM_E_INVAL, "n must be >= 1");
    hipLaunchKernelGGL(record_drafts_kernel, dim3(ceil_div(n, 256)), dim3(256), 0, (hipStream_t)stream,
                       (const int*)d_id, d_mask, (int*)d_draft_id, n);
    HIP_TRY(hipGetLastError());
    return DLLM_OK;
}

int dllm_quantize_q4_0(const void* d_src, int32_t src_dtype, int32_t rows, int32_t K, uint8_t* d_codes,
                       uint16_t* d_scales, dllm_stream stream) {
    if (!d_src || !d_codes || !d_scales) return fail(DLLM_E_INVAL, "NULL argument");
    if (rows < 1 || K < 1) return fail(DLLM_E_INVAL, "rows and K must be >= 1");
    if (src_dtype != DLLM_F32 && src_dtype != DLLM_BF16) return fail(DLLM_E_DTYPE, "source must be DLLM_F32 or DLLM_BF16");
    const long n = (long)rows * ceil_div(K, 32);
    const int blocks = ceil_div(n, 256);
    if (src_dtype == DLLM_F32)
        hipLaunchKernelGGL((quantize_q4_kernel<float>), dim3(blocks), dim3(256), 0, (hipStream_t)stream,
                           (const float*)d_src, rows, K, d_codes, d_scales);
    else
        hipLaunchKernelGGL((quantize_q4_kernel<uint16_t>), dim3(blocks), dim3(256), 0, (hipStream_t)stream,
                           (const uint16_t*)d_src, rows, K, d_codes, d_scales);
    HIP_TRY(hipGetLastError());
    return DLLM_OK;
}

int dllm_quantize_int8(const void* d_src, int32_t src_dtype, int32_t rows, int32_t K, int8_t* d_codes,
                       float* d_scales, dllm_stream stream) {
    if (!d_src || !d_codes || !d_scales) return fail(DLLM_E_INVAL, "NULL argument");
    if (rows < 1 || K < 1) return fail(DLLM_E_INVAL, "rows and K must be >= 1");
    if (src_dtype != DLLM_F32 && src_dtype != DLLM_BF16) return fail(DLLM_E_DTYPE, "source must be DLLM_F32 or DLLM_BF16");
    if (src_dtype == DLLM_F32)
        hipLaunchKernelGGL((quantize_i8_kernel<float>), dim3(rows), dim3(256), 0, (hipStream_t)stream,
                           (const float*)d_src, K, d_codes, d_scales);
    else
        hipLaunchKernelGGL((quantize_i8_kernel<uint16_t>), dim3(rows), dim3(256), 0, (hipStream_t)stream,
                           (const uint16_t*)d_src, K, d_codes, d_scales);
    HIP_TRY(hipGetLastError());
    return DLLM_OK;
}

int dllm_read_bandwidth(const void* d_buf, size_t bytes, uint32_t* d_sink, dllm_stream stream) {
    if (!d_buf || !d_sink) return fail(DLLM_E_INVAL, "NULL argument");
    if (((uintptr_t)d_buf & 15) != 0 || (bytes & 15) != 0)
        return fail(DLLM_E_INVAL, "buffer must be 16-byte aligned and a multiple of 16 bytes");
    if (bytes == 0) return DLLM_OK;
    hipLaunchKernelGGL(read_stream_kernel, dim3(8192), dim3(256), 0, (hipStream_t)stream, (const u32x4_t*)d_buf,
                       bytes / 16, d_sink);
    HIP_TRY(hipGetLastError());
    return DLLM_OK;
}

}  // extern "C"
