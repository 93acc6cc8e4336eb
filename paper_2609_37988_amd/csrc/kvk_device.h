// Device-side helpers of libkvk for gfx950: vector types, exact code unpacking,
// and the block layout of include/kvk.h (which the write kernel produces and the
// decode and dequantise kernels consume).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kvkd {

// Quantiser schemes (the values of kvk_qscheme), as template parameters.
constexpr int kQsKivi = 0, kQsSym = 1, kQsG64 = 2;

typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u2v __attribute__((ext_vector_type(2)));
typedef uint32_t u4v __attribute__((ext_vector_type(4)));

template <typename To, typename From>
__device__ __forceinline__ To bitcast(const From& x) {
  static_assert(sizeof(To) == sizeof(From), "size mismatch");
  return __builtin_bit_cast(To, x);
}

__device__ __forceinline__ half8 cat4(half2v a, half2v b, half2v c, half2v d) {
  u4v r = {bitcast<uint32_t>(a), bitcast<uint32_t>(b), bitcast<uint32_t>(c), bitcast<uint32_t>(d)};
  return bitcast<half8>(r);
}

__device__ __forceinline__ half2v h2(float a, float b) {
  half2v r = {(_Float16)a, (_Float16)b};
  return r;
}

__device__ __forceinline__ half2v h2s(float a) { return h2(a, a); }

// fp16 1024 + n has the integer n (n < 1024) in its low mantissa bits.
constexpr uint32_t kMagic = 0x64006400u;

// x in a VGPR, opaque to constant folding.  The asm is empty (no instruction): it
// only stops the compiler from folding a constant mask into a 32-bit literal,
// which the gfx9 VOP3 encoding cannot take (and_or would then become two VOP2
// instructions).  The compiler itself materialises the value (a v_mov it sees)
// and can hoist it out of loops.
__device__ __forceinline__ uint32_t in_vgpr(uint32_t x) {
  asm("" : "+v"(x));
  return x;
}

// (a & b) | c in one v_and_or_b32, selected by the compiler from C with the masks
// in registers.  Not inline assembly: the compiler's hazard checks do not look
// inside an asm statement, so an asm v_and_or_b32 that overwrote the accumulator
// input of an MFMA still in flight got no wait states and corrupted that product
// (seen in the 4-bit decode at d_h 64).
__device__ __forceinline__ uint32_t and_or(uint32_t a, uint32_t b, uint32_t c) {
  return (a & in_vgpr(b)) | in_vgpr(c);
}

// b = 4: one 32-bit chunk, slot s at bit 16*(s%2) + 4*(s/2).  Returns the 8 codes
// minus `off` as exact fp16 integers, slot pairs (0,1),(2,3),(4,5),(6,7).
// The and_or halves of the unpackers above without their fix-up: slot s holds
// 1024 + u_s / c_s exactly, with the slot factors c = raw_factors<BITS>() (powers
// of two).  A product over the slots then needs its other operand scaled by c and
// 1024 times that operand's slot sum taken off.
template <int BITS>
__device__ __forceinline__ half8 raw_codes(uint32_t w0, uint32_t w1) {
  if constexpr (BITS == 8) {
    const uint32_t M = 0x64646464u;
    return cat4(bitcast<half2v>(__builtin_amdgcn_perm(M, w0, 0x04010400u)),
                bitcast<half2v>(__builtin_amdgcn_perm(M, w0, 0x04030402u)),
                bitcast<half2v>(__builtin_amdgcn_perm(M, w1, 0x04010400u)),
                bitcast<half2v>(__builtin_amdgcn_perm(M, w1, 0x04030402u)));
  } else if constexpr (BITS == 4) {
    const uint32_t w8 = w0 >> 8;
    return cat4(bitcast<half2v>(and_or(w0, 0x000F000Fu, kMagic)), bitcast<half2v>(and_or(w0, 0x00F000F0u, kMagic)),
                bitcast<half2v>(and_or(w8, 0x000F000Fu, kMagic)), bitcast<half2v>(and_or(w8, 0x00F000F0u, kMagic)));
  } else {
    return cat4(bitcast<half2v>(and_or(w0, 0x00030003u, kMagic)), bitcast<half2v>(and_or(w0, 0x000C000Cu, kMagic)),
                bitcast<half2v>(and_or(w0, 0x00300030u, kMagic)), bitcast<half2v>(and_or(w0, 0x00C000C0u, kMagic)));
  }
}
template <int BITS>
__device__ __forceinline__ half8 raw_factors() {
  const _Float16 one = (_Float16)1.0f;
  if constexpr (BITS == 8) {
    return half8{one, one, one, one, one, one, one, one};
  } else if constexpr (BITS == 4) {
    const _Float16 s = (_Float16)0.0625f;
    return half8{one, one, s, s, one, one, s, s};
  } else {
    return half8{one, one, (_Float16)0.25f, (_Float16)0.25f, (_Float16)0.0625f, (_Float16)0.0625f,
                 (_Float16)0.015625f, (_Float16)0.015625f};
  }
}

__device__ __forceinline__ half8 unpack4(uint32_t w, float off) {
  const uint32_t w8 = w >> 8;
  half2v a = bitcast<half2v>(and_or(w, 0x000F000Fu, kMagic));   // 1024 + u
  half2v b = bitcast<half2v>(and_or(w, 0x00F000F0u, kMagic));   // 1024 + 16 u
  half2v c = bitcast<half2v>(and_or(w8, 0x000F000Fu, kMagic));
  half2v d = bitcast<half2v>(and_or(w8, 0x00F000F0u, kMagic));
  const half2v lo = h2s(-1024.0f - off);
  const half2v sx = h2s(0.0625f), hi = h2s(-64.0f - off);
  a = a + lo;
  c = c + lo;
  b = __builtin_elementwise_fma(b, sx, hi);  // (1024 + 16u)/16 - 64 - off, exact
  d = __builtin_elementwise_fma(d, sx, hi);
  return cat4(a, b, c, d);
}

// b = 2: one 32-bit word holds two chunks (even chunk at bits 2*(s/2), odd chunk
// 8 bits higher), slot s at bit 16*(s%2) + 2*(s/2) [+ 8].
__device__ __forceinline__ half8 unpack2_half(uint32_t w, float off) {
  half2v r[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const float scale = 1.0f / (float)(1 << (2 * v));
    half2v x = bitcast<half2v>(and_or(w, 0x00030003u << (2 * v), kMagic));  // 1024 + u*4^v
    r[v] = __builtin_elementwise_fma(x, h2s(scale), h2s(-1024.0f * scale - off));
  }
  return cat4(r[0], r[1], r[2], r[3]);
}

__device__ __forceinline__ void unpack2(uint32_t w, float off, half8& even, half8& odd) {
  even = unpack2_half(w, off);
  odd = unpack2_half(w >> 8, off);
}

// b = 8: two 32-bit words, slot s is byte s.
__device__ __forceinline__ half8 unpack8(uint32_t a, uint32_t b, float off) {
  const uint32_t M = 0x64646464u;
  const half2v lo = h2s(-1024.0f - off);
  half2v r0 = bitcast<half2v>(__builtin_amdgcn_perm(M, a, 0x04010400u)) + lo;
  half2v r1 = bitcast<half2v>(__builtin_amdgcn_perm(M, a, 0x04030402u)) + lo;
  half2v r2 = bitcast<half2v>(__builtin_amdgcn_perm(M, b, 0x04010400u)) + lo;
  half2v r3 = bitcast<half2v>(__builtin_amdgcn_perm(M, b, 0x04030402u)) + lo;
  return cat4(r0, r1, r2, r3);
}

// Cache policy of the loads that stream a compressed cache: non-temporal.  Each
// byte is read once per decode step, and on gfx950 a plain streaming read with
// this hint measured 7.1 TB/s against 6.3 TB/s without it.
constexpr int kStreamPolicy = 2;

// ---------------------------------------------------------------------------
// Cross-lane reductions without LDS round trips.
// ---------------------------------------------------------------------------

// Over the four 16-lane rows (lanes l % 16 + 16 k): v_permlane16_swap exchanges
// neighbouring rows and v_permlane32_swap the two halves of the wave; with both
// operands equal, each swap leaves a lane and its partner in the two results.
__device__ __forceinline__ float rows_max(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float rows_min(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fminf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fminf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float rows_sum(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// DPP lane permutation of x (CTRL: a DPP control word; every source lane valid).
template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
constexpr int kQuadXor1 = 0xB1;       // quad_perm [1,0,3,2]
constexpr int kQuadXor2 = 0x4E;       // quad_perm [2,3,0,1]
constexpr int kHalfRowMirror = 0x141; // lane i of each 8-lane half row <- lane 7 - i

// Over 8 consecutive lanes (8-aligned): two quad steps, then the half-row mirror
// pairs each quad with the other one.
__device__ __forceinline__ float max8(float x) {
  x = fmaxf(x, dpp<kQuadXor1>(x));
  x = fmaxf(x, dpp<kQuadXor2>(x));
  return fmaxf(x, dpp<kHalfRowMirror>(x));
}
__device__ __forceinline__ float sum8(float x) {
  x += dpp<kQuadXor1>(x);
  x += dpp<kQuadXor2>(x);
  return x + dpp<kHalfRowMirror>(x);
}

constexpr int kRowMirror = 0x140;  // lane i of each 16-lane row <- lane 15 - i

// Over 16 consecutive lanes (16-aligned): the 8-lane reduction, then the row mirror
// pairs each half row with the other one.
__device__ __forceinline__ float max16(float x) {
  x = max8(x);
  return fmaxf(x, dpp<kRowMirror>(x));
}
__device__ __forceinline__ float sum16(float x) {
  x = sum8(x);
  return x + dpp<kRowMirror>(x);
}

// ---------------------------------------------------------------------------
// Block layout (bytes from the start of a 32-token block).
// ---------------------------------------------------------------------------

__host__ __device__ inline int64_t block_bytes(int D, int bits, int kivi) {
  if (bits == 16) return 128LL * D;
  return kivi ? 8LL * D * (bits + 1) : 8LL * D * bits + 128;
}

// Byte of a part holding share byte o of lane lam, for P-byte lane shares: shares
// above 16 bytes are dealt out to the 64 lanes in 16-byte pieces.
__host__ __device__ inline int share_byte(int P, int lam, int o) {
  return P > 16 ? 1024 * (o >> 4) + 16 * lam + (o & 15) : lam * P + o;
}
// Inverse: the lane and share byte held at byte b of a part.
__host__ __device__ inline void share_of(int P, int b, int& lam, int& o) {
  if (P > 16) {
    lam = (b & 1023) >> 4;
    o = 16 * (b >> 10) + (b & 15);
  } else {
    lam = b / P;
    o = b % P;
  }
}

// Bit address of the K code of (token t, channel c) in a quantised block.
__device__ __forceinline__ int64_t k_code_bit(int D, int bits, int t, int c) {
  const int tau = t >> 4, i = t & 15, j = c >> 5, kg = (c & 31) >> 3, s = c & 7;
  const int lam = 16 * kg + i;
  const int64_t chunk = 2LL * D * bits * tau + share_byte(D * bits / 32, lam, j * bits);
  if (bits == 8) return 8 * chunk + 8 * s;
  if (bits == 4) return 8 * chunk + 16 * (s & 1) + 4 * (s >> 1);
  return 8 * (chunk - (j & 1) * 2) + 16 * (s & 1) + 2 * (s >> 1) + 8 * (j & 1);
}

// Bit address of the V code of (token t, channel c) in a quantised block.
__device__ __forceinline__ int64_t v_code_bit(int D, int bits, int t, int c) {
  const int i = c & 15, m = c >> 4, kg = (t & 15) >> 2, s = 4 * (t >> 4) + (t & 3);
  const int lam = 16 * kg + i;
  const int64_t chunk = 4LL * D * bits + share_byte(D * bits / 16, lam, m * bits);
  if (bits == 8) return 8 * chunk + 8 * s;
  if (bits == 4) return 8 * chunk + 16 * (s & 1) + 4 * (s >> 1);
  return 8 * (chunk - (m & 1) * 2) + 16 * (s & 1) + 2 * (s >> 1) + 8 * (m & 1);
}

// Byte address of the bf16 K / V value of (t, c) in a bf16 block.
__device__ __forceinline__ int k_bf16_byte(int D, int t, int c) {
  const int tau = t >> 4, i = t & 15, j = c >> 5, kg = (c & 31) >> 3, s = c & 7;
  return 32 * D * tau + share_byte(D / 2, 16 * kg + i, 16 * j) + 2 * s;
}
__device__ __forceinline__ int v_bf16_byte(int D, int t, int c) {
  const int i = c & 15, m = c >> 4, kg = (t & 15) >> 2, s = 4 * (t >> 4) + (t & 3);
  return 64 * D + share_byte(D, 16 * kg + i, 16 * m) + 2 * s;
}

// Index (in fp16 units) of the KIVI32 V-meta entry w (0 scale, 1 zero) of
// (token t, channel group g).
__device__ __forceinline__ int v_meta_index(int t, int g, int w) {
  const int kg = (t & 15) >> 2, s = 4 * (t >> 4) + (t & 3);
  return ((g * 2 + w) * 4 + kg) * 8 + s;
}

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float((uint32_t)b << 16);
}

__device__ __forceinline__ uint16_t f32_to_bf16_bits(float x) {
  __bf16 h = (__bf16)x;  // round to nearest even
  return bitcast<uint16_t>(h);
}

__device__ __forceinline__ float f16_bits_to_f32(uint16_t b) {
  return (float)bitcast<_Float16>(b);
}

}  // namespace kvkd
