// Device-side building blocks shared by the dprc kernels (gfx950 / CDNA4).
//
//  * Philox4x32-10 (Salmon et al., SC'11) and the probe / noise streams;
//  * bf16 <-> fp32 conversions and the hi/lo split of an fp32 value into two
//    bf16 values (operands of the bf16 matrix cores);
//  * wrappers for the bf16 MFMA with K = 32 and for the LDS transpose read.
//
// Lane layouts used below (wave64, checked on gfx950):
//  mfma 16x16x32 bf16  A[16x32]: lane l holds A[l%16][8*(l/16) + j], j = 0..7
//                      B[32x16]: lane l holds B[8*(l/16) + j][l%16]
//                      D[16x16]: lane l holds D[4*(l/16) + i][l%16], i = 0..3
//  ds_read_tr16_b64    within each 16-lane group, lane 4r+c passes the address
//                      of 4 consecutive 16-bit elements (row r of a 4x16
//                      block, columns 4c..4c+3); lane j of the group receives
//                      column j of the 4 rows.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dprc {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef __attribute__((address_space(3))) bf16x4_t lds_bf16x4_t;

struct u32x4 {
  uint32_t x, y, z, w;
};

// ---- Philox4x32-10 -----------------------------------------------------------
__device__ __forceinline__ u32x4 philox4x32_10(u32x4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    if (round) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint32_t a = c.x, b = c.z;
    const uint32_t lo0 = 0xD2511F53u * a, hi0 = __umulhi(0xD2511F53u, a);
    const uint32_t lo1 = 0xCD9E8D57u * b, hi1 = __umulhi(0xCD9E8D57u, b);
    c = u32x4{hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0};
  }
  return c;
}

enum : uint32_t { kStreamProbe = 0, kStreamSketch = 1, kStreamNoise = 2, kStreamGaussProbe = 3 };
enum : int { kProbeRademacher = 0, kProbeHadamard = 1 };

// Four consecutive probe words (rows 128*blk .. 128*blk+127) of column j.
__device__ __forceinline__ u32x4 rademacher_block(uint32_t key0, uint32_t key1, uint32_t layer,
                                                  uint32_t stream, uint32_t blk, uint32_t col) {
  return philox4x32_10(u32x4{blk, col, layer, stream}, key0, key1);
}

// Word w (rows 32w .. 32w+31) of column j of the Sylvester-Hadamard sign pattern.  The
// sign of entry (r, j) is the parity of popcount(r & j).  Within a word, bit k of r
// (k < 5) follows a fixed 32-bit pattern, so the word is the XOR of the patterns of the set
// bits of j & 31, inverted when popcount(32 w & j) is odd.
__device__ __forceinline__ uint32_t hadamard_word(uint32_t w, uint32_t col) {
  constexpr uint32_t kBitPattern[5] = {0xAAAAAAAAu, 0xCCCCCCCCu, 0xF0F0F0F0u, 0xFF00FF00u, 0xFFFF0000u};
  uint32_t pat = 0;
#pragma unroll
  for (int k = 0; k < 5; ++k) pat ^= ((col >> k) & 1u) ? kBitPattern[k] : 0u;
  return (__popc((w << 5) & col) & 1) ? ~pat : pat;
}

__device__ __forceinline__ uint32_t tail_mask(int64_t m, int64_t w) {
  const int64_t rem = m - 32 * w;
  return rem >= 32 ? 0xFFFFFFFFu : (rem <= 0 ? 0u : ((1u << rem) - 1u));
}

// ---- bf16 ----------------------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

// round to nearest even; NaN stays NaN
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (u >> 16) | 0x40u;
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

// f = hi + lo + O(2^-17 |f|), both bf16
__device__ __forceinline__ void split_bf16(float f, uint32_t& hi, uint32_t& lo) {
  hi = f32_to_bf16(f);
  lo = f32_to_bf16(f - bf16_to_f32(hi));
}

// 8 signs (bit set -> -1) to 8 bf16 values +-1 packed in four dwords
__device__ __forceinline__ uint4 signs_to_bf16x8(uint32_t byte) {
  uint4 r;
  r.x = 0x3F803F80u | ((byte & 1u) << 15) | ((byte & 2u) << 30);
  r.y = 0x3F803F80u | ((byte & 4u) << 13) | ((byte & 8u) << 28);
  r.z = 0x3F803F80u | ((byte & 16u) << 11) | ((byte & 32u) << 26);
  r.w = 0x3F803F80u | ((byte & 64u) << 9) | ((byte & 128u) << 24);
  return r;
}

// Loads of 8 consecutive bf16 of a token row.  The fast form is one 16-byte
// load with no branch: callers pass a pointer that is valid and 16-byte aligned
// even when the lane is masked (a clamped address) and the value is zeroed by a
// select, so all loads of a stage stay in flight together.  The element form
// serves rows that are not 16-byte aligned or widths that are not a multiple
// of 8 (the host picks the form per launch).
__device__ __forceinline__ uint4 load8_sel(const uint16_t* p, bool ok) {
  const uint4 v = *reinterpret_cast<const uint4*>(p);
  return ok ? v : uint4{0, 0, 0, 0};
}

__device__ __forceinline__ uint4 load8_elem(const uint16_t* row, int64_t u, int64_t lim, bool ok) {
  uint32_t h[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) h[j] = (ok && u + j < lim) ? (uint32_t)row[u + j] : 0u;
  return uint4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
}

// Raw buffer resource over [base, base + bytes): a load at a byte offset at or
// beyond `bytes` returns zero without touching memory (hardware range check), so
// masked lanes need no branch, only an out-of-range offset.  bytes < 2^31; base
// and bytes are wave-uniform (the resource lives in scalar registers; reading the
// byte count through readfirstlane keeps a value that the compiler computed in a
// vector register from turning every load into a loop over lanes).
constexpr uint32_t kOobOffset = 0x80000000u;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0,
                                           (int)__builtin_amdgcn_readfirstlane(bytes), 0x00020000);
}
__device__ __forceinline__ uint4 buffer_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0));
}
// The same load marked non-temporal (cache policy NT): for operands streamed once, whose
// lines need not stay in the caches.  A read-only probe over the stack workload's 54.7 GB
// streamed 6.6 to 6.7 TB/s with it against 5.9 to 6.2 TB/s without.
constexpr int kCachePolicyNT = 2;
__device__ __forceinline__ uint4 buffer_load16_nt(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, kCachePolicyNT));
}

// The 8 bf16 values +-1 of one byte of probe signs (bit set -> -1) as a 16x16x32
// B operand fragment.  `P` holds the byte in bits 0..7 of both 16-bit halves
// (bits 8..15 of each half are ignored); `mask` = 0x80008000 and `one` =
// 0x3F803F80 for a probe column, both 0 for a column that takes zeros.  Dword j
// gets bit 2j into the sign of its low bf16 and bit 2j+1 into the sign of its high
// bf16: a packed 16-bit shift left moves both into bit 15 of their halves.
typedef unsigned short u16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t shl16x2(uint32_t v, unsigned short lo, unsigned short hi) {
  return __builtin_bit_cast(uint32_t, __builtin_bit_cast(u16x2_t, v) << u16x2_t{lo, hi});
}
__device__ __forceinline__ uint4 expand_signs(uint32_t P, uint32_t mask, uint32_t one) {
  return uint4{(shl16x2(P, 15, 14) & mask) | one, (shl16x2(P, 13, 12) & mask) | one,
               (shl16x2(P, 11, 10) & mask) | one, (shl16x2(P, 9, 8) & mask) | one};
}

template <bool FAST>
__device__ __forceinline__ uint4 load_bf16x8(const uint16_t* row, int64_t u, int64_t lim, bool row_ok,
                                             const uint16_t* safe) {
  if constexpr (FAST) {
    const bool ok = row_ok && u < lim;          // lim % 8 == 0: u < lim implies u + 8 <= lim
    return load8_sel(ok ? row + u : safe, ok);
  } else {
    return load8_elem(row, u, lim, row_ok);
  }
}

// ---- matrix cores and LDS ------------------------------------------------------------
__device__ __forceinline__ f32x4_t mfma16x16x32(const uint4& a, const uint4& b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                  __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

__device__ __forceinline__ uint2 lds_read_tr16(const uint16_t* p) {
  bf16x4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)(p));
  return __builtin_bit_cast(uint2, v);
}

__device__ __forceinline__ uint4 make_u4(uint2 a, uint2 b) { return uint4{a.x, a.y, b.x, b.y}; }

// component-wise select (a select of whole vectors can end up as a select of
// their stack addresses)
__device__ __forceinline__ uint4 select4(bool c, const uint4& a, const uint4& b) {
  return uint4{c ? a.x : b.x, c ? a.y : b.y, c ? a.z : b.z, c ? a.w : b.w};
}

// Two standard normals from two Philox words (Box-Muller): uniforms
// (floor(x / 2^9) + 1/2) * 2^-23, exact in fp32 and never 0 or 1.
__device__ __forceinline__ void box_muller(uint32_t x0, uint32_t x1, float& n0, float& n1) {
  const float u1 = ((float)(x0 >> 9) + 0.5f) * 0x1p-23f;
  const float u2 = ((float)(x1 >> 9) + 0.5f) * 0x1p-23f;
  const float r = sqrtf(-2.f * logf(u1));
  float sn, cs;
  sincospif(2.f * u2, &sn, &cs);
  n0 = r * cs;
  n1 = r * sn;
}

// c = min(1, C / sqrt(n)) for a summed squared-norm estimate n (Algorithm 1);
// n = 0 gives 1, a NaN, negative or infinite n gives 0.
__device__ __forceinline__ float clip_factor(float n, float C) {
  if (!(n >= 0.f) || isinf(n)) return 0.f;
  if (n <= C * C) return 1.f;
  return C / sqrtf(n);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

}  // namespace dprc
