// Shared device helpers for the gfx950 denoising-step kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));

namespace dllm {

// Weight element types of the packed GEMM operand.
enum WType : int { WT_F32 = 0, WT_BF16 = 1, WT_I8 = 2, WT_Q4 = 3 };

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7F800000u) == 0x7F800000u) return (uint16_t)((u >> 16) | ((u & 0xFFFFu) ? 0x40u : 0u));
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

template <typename T> __device__ __forceinline__ float to_f32(T v);
template <> __device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f32<uint16_t>(uint16_t v) { return bf16_to_f32(v); }

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ uint16_t from_f32<uint16_t>(float v) { return f32_to_bf16(v); }

// ---------------------------------------------------------------------------
// MFMA operand fragments (gfx950, wave64)
//
// v_mfma_f32_16x16x32_bf16: lane l (g = l / 16) holds A[l % 16][8g .. 8g+7] and
// B[8g .. 8g+7][l % 16]; the result lane l holds D[4g + i][l % 16], i = 0..3.
// v_mfma_f32_16x16x4_f32:   lane l holds A[l % 16][g] and B[g][l % 16].
//
// A "chunk" is 16 rows x KC columns stored as 64 lanes x 16 bytes (1 KiB):
//   bf16 (KC = 32): lane l bytes = row l%16, cols 8g .. 8g+7
//   f32  (KC = 16): lane l float s = row l%16, col 4s + g (s = 0..3, one MFMA each)
//   int8 (KC = 64): lane l byte 8h + e = row l%16, col 32h + 8g + e (h = 0..1)
//   Q4_0 (KC = 64, 512-byte chunks, 8 bytes per lane): dword h (= 32-column block
//        h) of lane l holds the 4-bit codes of row l%16, cols 32h + 8g + e, e = 0..7,
//        code e at bits 4 * (e / 2) (e even) or 16 + 4 * (e / 2) (e odd), so that
//        one shift-and-mask yields two bf16 values of adjacent columns (q4_unpack);
//        the chunk's fp16 scales sit in a separate array, 16 rows x 2 blocks.
// Packed weights: chunk (nt, kc) at byte ((nt * KCn + kc) * 64 + lane) * 16
// (Q4_0: * 8).
//
// Activation fragments use the same chunk shape with rows = tokens.  For fp32
// models a chunk holds 16 fp32 columns.  For bf16 / int8-weight models a value v
// is carried as two bf16 planes, hi = bf16(v) and lo = bf16(v - hi), so that the
// A operand keeps ~16 significant bits; a chunk is then 32 columns, hi plane
// (1 KiB) followed by lo plane (1 KiB), and the GEMM issues one MFMA per plane.
//   fp32:  chunk (mt, kcx) at byte (mt * KCx + kcx) * 1024
//   hi/lo: chunk (mt, kcx) at byte (mt * KCx + kcx) * 2048 (+1024 for lo)
// ---------------------------------------------------------------------------

template <int WT> struct WTraits;
template <> struct WTraits<WT_F32> { static constexpr int KC = 16; static constexpr int XPER = 1; };
template <> struct WTraits<WT_BF16> { static constexpr int KC = 32; static constexpr int XPER = 1; };
template <> struct WTraits<WT_I8> { static constexpr int KC = 64; static constexpr int XPER = 2; };
template <> struct WTraits<WT_Q4> { static constexpr int KC = 64; static constexpr int XPER = 2; };

// Bytes of one packed weight chunk (16 rows x KC columns).
template <int WT> constexpr int wchunk_bytes() { return WT == WT_Q4 ? 512 : 1024; }

// Bytes of one activation chunk.
template <bool F32> struct XChunk { static constexpr int bytes = F32 ? 1024 : 2048; };

// hi / lo bf16 split of an fp32 value.
__device__ __forceinline__ void split_bf16(float v, uint16_t& hi, uint16_t& lo) {
    hi = f32_to_bf16(v);
    lo = f32_to_bf16(v - bf16_to_f32(hi));
}

// Store activation element (m, k) into the fragment buffer with KCx chunks per tile row.
template <bool F32>
__device__ __forceinline__ void xfrag_store(void* base, int m, int k, int KCx, float v) {
    const int mt = m >> 4, r = m & 15;
    if (F32) {
        const int kc = k >> 4, kk = k & 15;
        const int g = kk & 3, s = kk >> 2;
        char* p = (char*)base + ((size_t)(mt * KCx + kc) * 64 + (r + 16 * g)) * 16 + s * 4;
        *(float*)p = v;
    } else {
        const int kc = k >> 5, kk = k & 31;
        const int g = kk >> 3, e = kk & 7;
        char* p = (char*)base + (size_t)(mt * KCx + kc) * 2048 + (r + 16 * g) * 16 + e * 2;
        uint16_t hi, lo;
        split_bf16(v, hi, lo);
        *(uint16_t*)p = hi;
        *(uint16_t*)(p + 1024) = lo;
    }
}

// Store four consecutive activation columns k .. k+3 (k % 4 == 0) of row m.
template <bool F32>
__device__ __forceinline__ void xfrag_store4(void* base, int m, int k, int KCx, float4 v) {
    if (F32) {
        xfrag_store<true>(base, m, k + 0, KCx, v.x);
        xfrag_store<true>(base, m, k + 1, KCx, v.y);
        xfrag_store<true>(base, m, k + 2, KCx, v.z);
        xfrag_store<true>(base, m, k + 3, KCx, v.w);
    } else {
        const int mt = m >> 4, r = m & 15;
        const int kc = k >> 5, kk = k & 31;
        const int g = kk >> 3, e = kk & 7;     // e is 0 or 4
        char* p = (char*)base + (size_t)(mt * KCx + kc) * 2048 + (r + 16 * g) * 16 + e * 2;
        uint16_t h[4], l[4];
        split_bf16(v.x, h[0], l[0]);
        split_bf16(v.y, h[1], l[1]);
        split_bf16(v.z, h[2], l[2]);
        split_bf16(v.w, h[3], l[3]);
        *(uint2*)p = make_uint2(h[0] | ((uint32_t)h[1] << 16), h[2] | ((uint32_t)h[3] << 16));
        *(uint2*)(p + 1024) = make_uint2(l[0] | ((uint32_t)l[1] << 16), l[2] | ((uint32_t)l[3] << 16));
    }
}

__device__ __forceinline__ f32x4_t mfma_bf16(const u32x4_t& a, const u32x4_t& b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                  __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

// v_mfma_f32_16x16x32_f16: the same operand layout with fp16 elements.
__device__ __forceinline__ f32x4_t mfma_f16(const u32x4_t& a, const u32x4_t& b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, a), __builtin_bit_cast(f16x8_t, b), c,
                                                 0, 0, 0);
}

__device__ __forceinline__ f32x4_t mfma_f32(float a, float b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// 8 signed bytes (two dwords) -> 8 bf16 (exact: |q| <= 127 fits the 8-bit significand).
__device__ __forceinline__ u32x4_t i8x8_to_bf16x8(uint32_t lo, uint32_t hi) {
    u32x4_t r;
    uint32_t w[2] = {lo, hi};
#pragma unroll
    for (int j = 0; j < 2; ++j) {
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            const int b0 = (int)(int8_t)((w[j] >> (16 * p)) & 0xFF);
            const int b1 = (int)(int8_t)((w[j] >> (16 * p + 8)) & 0xFF);
            // the high halves of the two floats (exact: |b| <= 128 needs 8 bits), packed
            // by one byte permute: bytes 2-3 of f0, then bytes 2-3 of f1
            const uint32_t f0 = __float_as_uint((float)b0);
            const uint32_t f1 = __float_as_uint((float)b1);
            r[2 * j + p] = __builtin_amdgcn_perm(f1, f0, 0x07060302u);
        }
    }
    return r;
}

// Q4_0: four dwords of bf16 pairs (128 + q) for the 8 codes of one dword (see the
// chunk layout above); 128 + q is exact in bf16 (7 stored significand bits).
__device__ __forceinline__ u32x4_t q4_unpack(uint32_t c) {
    // the mask and the bf16 128 bias kept in registers (the empty asm statements hide
    // their values), so that each dword is one v_and_or_b32 after its shift: a
    // 3-operand VALU instruction takes no literal here, and with literals the compiler
    // emitted a separate AND and OR (LLaDA-8B Q4_0 step 3.22 -> 3.13 ms)
    uint32_t mask = 0x000F000Fu, bias = 0x43004300u;
    asm("" : "+s"(mask));
    asm("" : "+v"(bias));
    u32x4_t r;
#pragma unroll
    for (int i = 0; i < 4; ++i) r[i] = ((c >> (4 * i)) & mask) | bias;
    return r;
}

__device__ __forceinline__ float f16_bits_to_f32(uint32_t h) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)h);
}

__device__ __forceinline__ uint16_t f32_to_f16_bits(float f) {
    return __builtin_bit_cast(uint16_t, (_Float16)f);    // round to nearest even
}

// fp16 cache values: round to nearest even, saturated to the largest finite fp16.
__device__ __forceinline__ uint16_t f16_sat(float v) { return f32_to_f16_bits(fminf(fmaxf(v, -65504.f), 65504.f)); }

// hi / lo fp16 split (an fp16 MFMA operand with ~21 significant bits): hi = fp16(v),
// lo = fp16(v - hi), both saturated.
__device__ __forceinline__ void split_f16(float v, uint16_t& hi, uint16_t& lo) {
    v = fminf(fmaxf(v, -65504.f), 65504.f);
    hi = f32_to_f16_bits(v);
    lo = f32_to_f16_bits(v - f16_bits_to_f32(hi));
}

// Q4_0 decision for one block of 32 columns [k0, k0 + 32) of a row (columns >= K
// read as 0), in fp32: m = the value of largest magnitude (first in column order),
// d = m / -8, inv = 1 / d (0 when d = 0).  A value x gets code min(15, trunc(x * inv + 8.5)).
template <typename ST>
__device__ __forceinline__ void q4_block(const ST* row, int k0, int K, float& d, float& inv) {
    float amax = 0.f, m = 0.f;
    for (int k = k0; k < k0 + 32; ++k) {
        const float x = (k < K) ? to_f32<ST>(row[k]) : 0.f;
        if (fabsf(x) > amax) { amax = fabsf(x); m = x; }
    }
    d = __fdiv_rn(m, -8.0f);
    inv = (d != 0.f) ? __fdiv_rn(1.0f, d) : 0.f;
}

// The product and the sum are rounded separately (no fused multiply-add), as the
// format's reference arithmetic does: a fused x * inv + 8.5 moves codes that sit on a
// rounding boundary.
__device__ __forceinline__ uint32_t q4_code(float x, float inv) {
#pragma clang fp contract(off)
    const float p = x * inv;
    const int q = (int)(p + 8.5f);
    return (uint32_t)min(15, q);
}

__device__ __forceinline__ float warp_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}
__device__ __forceinline__ float warp_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
    return v;
}

__device__ __forceinline__ u32x4_t ldg16(const void* p) { return *(const u32x4_t*)p; }
__device__ __forceinline__ u32x4_t ldg16_nt(const void* p) {
    return __builtin_nontemporal_load((const u32x4_t*)p);
}
__device__ __forceinline__ u32x2_t ldg8_nt(const void* p) {
    return __builtin_nontemporal_load((const u32x2_t*)p);
}

}  // namespace dllm
