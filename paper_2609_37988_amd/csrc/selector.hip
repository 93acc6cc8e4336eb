// The selector's forward pass (KV-Kaizen §2.3, App. B "Selector architecture"): a
// prompt's token embeddings -> a linear map to width 256 -> two bidirectional
// pre-norm transformer blocks (RMSNorm, 4 heads of 64 with rotary embeddings on q
// and k, RMSNorm, SwiGLU of inner width 1024; residuals around both sublayers) ->
// a final RMSNorm -> time average -> optional budget scale and shift (FiLM) -> one
// linear head per layer -> argmax action per layer (the depth action masked at the
// first layer, or everywhere when depth is not in the action space).  It runs once
// per prompt at prefill; the plan it yields is held for the whole generation.
// Weights are inputs (packed bf16, layout in include/kvk.h).
//
// Kernels (T = prompt length):
//   sel_rope_kernel: the rotation table cos/sin(t * theta_i), t < T, i < 32, formed
//       in fp64 and stored fp32 (the angles reach 3e4 rad; an fp32 product would
//       put errors of 1e-3 rad into them).
//   sel_gemm_kernel<EPI>: C = A [T, K] . W^T, W [N, K] (bf16 operands on MFMA
//       16x16x32, fp32 accumulation); 64 x 256 output tiles per workgroup, the A and
//       W rows of each k-step staged in LDS (double-buffered); by EPI the epilogue
//       stores fp32, adds into the fp32 residual stream, forms SiLU(gate) * up to
//       bf16 (the W rows of a tile are mapped so that a lane holds a gate column and
//       its up column), or rotates q and k (a lane holds channel i and i + 32 of a
//       head) and splits q, k (bf16 rows) and v (bf16, transposed per head for the
//       attention's value operand).
//   sel_rmsnorm_kernel: one wave per row of 256, fp32 in, bf16 out.
//   sel_attention_kernel: bidirectional attention, 4 heads of 64; a workgroup takes
//       128 queries of one head (4 waves x two 16-query tiles) and walks the keys
//       in tiles of 64, double-buffered in LDS; S^T = K Q^T, one online-softmax
//       step (base 2) per query and tile, O^T += V^T P^T with P^T taken straight
//       from the S^T accumulators (the key order of the product's k-slots follows
//       the accumulator layout), the probability sums on MFMA as well; on short
//       prompts the keys split across workgroups too, and sel_attn_merge_kernel
//       combines the splits.
//   sel_pool_kernel / sel_heads_kernel: the final RMSNorm and the time average
//       (per-chunk partial sums of the normalised rows, then their sum), the budget
//       scale and shift, the per-layer logits and the argmax (a workgroup per layer).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <type_traits>

#include "kvk_device.h"
#include "kvk_internal.h"

using namespace kvkd;

namespace {

constexpr int kW = 256, kHeads = 4, kDh = 64, kFfn = 1024, kMaxActions = 32;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kRmsEps = 1e-6f;
constexpr double kRopeBase = 10000.0;
constexpr int kRec = kDh + 4;  // key-split record: 64 outputs, max, sum, 2 pad (16-byte rows)

__device__ __forceinline__ f4 mfma_bf(bf16x8 a, bf16x8 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float silu(float x) { return x / (1.0f + __expf(-x)); }

// cs[t][i] = (cos, sin)(t * base^(-i/32)), i < 32: the rotate-half pair (i, i + 32)
// of every head turns by that angle at position t.
__global__ __launch_bounds__(256) void sel_rope_kernel(float2* cs, int T) {
  const int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (k >= (int64_t)T * (kDh / 2)) return;
  const int i = (int)(k % (kDh / 2));
  const double theta = pow(kRopeBase, -(double)i / (kDh / 2));
  double s, c;
  sincos((double)(k / (kDh / 2)) * theta, &s, &c);
  cs[k] = make_float2((float)c, (float)s);
}

enum Epi { kStoreF32 = 0, kAddF32 = 1, kSwiGlu = 2, kQkv = 3 };

struct GemmArgs {
  const uint16_t* a;   // [M][K] bf16
  const uint16_t* w;   // [N][K] bf16 (kSwiGlu: gate rows [1024][K], then up rows)
  float* out_f32;      // [M][N] (kStoreF32, kAddF32)
  uint16_t* out_bf16;  // [M][1024] (kSwiGlu), [M][512] q|k (kQkv)
  uint16_t* vt;        // kQkv: [heads][64][vt_pitch] values, transposed
  const float2* rope;  // kQkv: [M][32] cos, sin
  float* part;         // split-K: [gridDim.z][M][N] raw partial sums (no epilogue); else null
  int32_t M, N, K, vt_pitch;
  int32_t k_len;       // k per split (a multiple of 32)
};

// Workgroup tile: 64 rows of C x 256 columns (N % 256 == 0, K % 32 == 0), wave w
// takes columns 64 w .. + 63 of all 64 rows (4 x 4 MFMA tiles).  Per k-step of 32 the
// A rows and W rows of the tile are staged in LDS (double-buffered: the next step's
// share of each thread is loaded into registers while the current step is consumed,
// one barrier per step); lane (row i16, k-group kg) feeds 8 consecutive k.
// kSwiGlu: tile y covers hidden columns 128 y .. + 127; wave w's MFMA tiles j = 0, 1
// read gate rows 128 y + 32 w + 16 j + i and tiles j = 2, 3 the up rows of the same
// hidden columns, so acc[i][j] and acc[i][j + 2] of a lane hold a gate and its up.
template <int EPI>
__global__ __launch_bounds__(256) void sel_gemm_kernel(GemmArgs g) {
  constexpr int BM = 64, BN = 256, KP = 32 + 8;  // LDS row pitch (halfs)
  __shared__ uint16_t as[2][BM][KP];
  __shared__ uint16_t bs[2][BN][KP];
  const int tid = threadIdx.x, lane = tid & 63, i16 = lane & 15, kg = lane >> 4, wv = tid >> 6;
  const int r0 = blockIdx.x * BM, c0 = blockIdx.y * BN;
  // staging share: A row tid / 4 and LDS W rows tid / 4 + 64 r, 8 k at 8 (tid % 4)
  const int sr = tid >> 2, sk = 8 * (tid & 3);
  const bool a_ok = r0 + sr < g.M;
  const uint16_t* ap = g.a + (int64_t)(a_ok ? r0 + sr : 0) * g.K + sk;
  int64_t wrow0, wrstep;  // W row of LDS row sr + 64 r: wrow0 + r * wrstep
  if constexpr (EPI == kSwiGlu) {
    wrow0 = (sr < 32 ? 0 : kFfn - 32) + blockIdx.y * 128 + sr;
    wrstep = 32;
  } else {
    wrow0 = c0 + sr;
    wrstep = 64;
  }
  const uint16_t* wp = g.w + wrow0 * g.K + sk;
  const int64_t wstep = wrstep * g.K;
  uint4 areg, w0, w1, w2, w3;
  auto fetch = [&](int k0) {
    areg = a_ok ? *reinterpret_cast<const uint4*>(ap + k0) : make_uint4(0, 0, 0, 0);
    w0 = *reinterpret_cast<const uint4*>(wp + k0);
    w1 = *reinterpret_cast<const uint4*>(wp + wstep + k0);
    w2 = *reinterpret_cast<const uint4*>(wp + 2 * wstep + k0);
    w3 = *reinterpret_cast<const uint4*>(wp + 3 * wstep + k0);
  };
  auto stash = [&](int buf) {
    *reinterpret_cast<uint4*>(&as[buf][sr][sk]) = areg;
    *reinterpret_cast<uint4*>(&bs[buf][sr][sk]) = w0;
    *reinterpret_cast<uint4*>(&bs[buf][sr + 64][sk]) = w1;
    *reinterpret_cast<uint4*>(&bs[buf][sr + 128][sk]) = w2;
    *reinterpret_cast<uint4*>(&bs[buf][sr + 192][sk]) = w3;
  };
  f4 acc[4][4] = {};
  const int kb = blockIdx.z * g.k_len, ke = min(g.K, kb + g.k_len);  // this split's k range
  fetch(kb);
  stash(0);
  __syncthreads();
  int buf = 0;
  for (int k0 = kb; k0 < ke; k0 += 32, buf ^= 1) {
    const bool more = k0 + 32 < ke;  // uniform
    if (more) fetch(k0 + 32);
    bf16x8 av[4], wv8[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      av[i] = *reinterpret_cast<const bf16x8*>(&as[buf][16 * i + i16][8 * kg]);
      wv8[i] = *reinterpret_cast<const bf16x8*>(&bs[buf][64 * wv + 16 * i + i16][8 * kg]);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = mfma_bf(wv8[j], av[i], acc[i][j]);  // C^T tile: rows n, cols m
    if (more) stash(buf ^ 1);  // that buffer was last read before the previous barrier
    __syncthreads();
  }
  // acc[i][j]: lane (m = r0 + 16 i + i16) holds LDS column 64 wv + 16 j + 4 kg + e
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = r0 + 16 * i + i16;
    if (m >= g.M) continue;
    if constexpr (EPI == kSwiGlu) {
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int hc = blockIdx.y * 128 + 32 * wv + 16 * j + 4 * kg;  // hidden column
        uint2 w2;
        w2.x = (uint32_t)f32_to_bf16_bits(silu(acc[i][j][0]) * acc[i][j + 2][0]) |
               ((uint32_t)f32_to_bf16_bits(silu(acc[i][j][1]) * acc[i][j + 2][1]) << 16);
        w2.y = (uint32_t)f32_to_bf16_bits(silu(acc[i][j][2]) * acc[i][j + 2][2]) |
               ((uint32_t)f32_to_bf16_bits(silu(acc[i][j][3]) * acc[i][j + 2][3]) << 16);
        *reinterpret_cast<uint2*>(g.out_bf16 + (int64_t)m * kFfn + hc) = w2;
      }
      continue;
    }
    if constexpr (EPI == kQkv) {
      if (c0 < 2 * kW) {  // q or k of head wv: rotate pairs (c, c + 32), c = 16 j + 4 kg + e
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float2 r = g.rope[(int64_t)m * (kDh / 2) + 16 * j + 4 * kg + e];
            const float x1 = acc[i][j][e], x2 = acc[i][j + 2][e];
            acc[i][j][e] = x1 * r.x - x2 * r.y;
            acc[i][j + 2][e] = x2 * r.x + x1 * r.y;
          }
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n0 = c0 + 64 * wv + 16 * j + 4 * kg;
      if (g.part) {  // split-K: the reduce kernel applies the epilogue
        *reinterpret_cast<f4*>(g.part + ((int64_t)blockIdx.z * g.M + m) * g.N + n0) = acc[i][j];
        continue;
      }
      const f4 v = acc[i][j];
      if constexpr (EPI == kStoreF32) {
        *reinterpret_cast<f4*>(g.out_f32 + (int64_t)m * g.N + n0) = v;
      } else if constexpr (EPI == kAddF32) {
        f4* px = reinterpret_cast<f4*>(g.out_f32 + (int64_t)m * g.N + n0);
        *px = *px + v;
      } else if (n0 < 2 * kW) {  // q, k rows (the 4 columns never straddle 512)
        uint2 w2;
        w2.x = (uint32_t)f32_to_bf16_bits(v[0]) | ((uint32_t)f32_to_bf16_bits(v[1]) << 16);
        w2.y = (uint32_t)f32_to_bf16_bits(v[2]) | ((uint32_t)f32_to_bf16_bits(v[3]) << 16);
        *reinterpret_cast<uint2*>(g.out_bf16 + (int64_t)m * (2 * kW) + n0) = w2;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) g.vt[(int64_t)(n0 + e - 2 * kW) * g.vt_pitch + m] = f32_to_bf16_bits(v[e]);
      }
    }
  }
}

// Split-K epilogue for the fp32 outputs (N = 256): out[m][n] (+)= sum over the splits
// of part[s][m][n], in split order.  One thread per 4 columns.
template <int EPI>
__global__ __launch_bounds__(256) void sel_splitk_kernel(const float* part, int splits, float* out, int M) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;  // f4 index
  if (i >= (int64_t)M * (kW / 4)) return;
  f4 v = *reinterpret_cast<const f4*>(part + 4 * i);
  for (int sp = 1; sp < splits; ++sp) v += *reinterpret_cast<const f4*>(part + (int64_t)sp * M * kW + 4 * i);
  f4* po = reinterpret_cast<f4*>(out + 4 * i);
  if constexpr (EPI == kAddF32) *po = *po + v;
  else *po = v;
}

__device__ __forceinline__ float wave_sum(float s) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off);
  return s;
}

// One wave per row of 256: RMSNorm (eps 1e-6, gain) to bf16.
__global__ __launch_bounds__(256) void sel_rmsnorm_kernel(const float* x, const uint16_t* gain, uint16_t* out,
                                                          int M) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  const f4 v = *reinterpret_cast<const f4*>(x + (int64_t)row * kW + 4 * lane);
  const float ms = wave_sum(v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3]) * (1.0f / kW);
  const float rs = 1.0f / sqrtf(ms + kRmsEps);
  uint2 w2;
  const int c = 4 * lane;
  w2.x = (uint32_t)f32_to_bf16_bits(v[0] * rs * bf16_to_f32(gain[c])) |
         ((uint32_t)f32_to_bf16_bits(v[1] * rs * bf16_to_f32(gain[c + 1])) << 16);
  w2.y = (uint32_t)f32_to_bf16_bits(v[2] * rs * bf16_to_f32(gain[c + 2])) |
         ((uint32_t)f32_to_bf16_bits(v[3] * rs * bf16_to_f32(gain[c + 3])) << 16);
  *reinterpret_cast<uint2*>(out + (int64_t)row * kW + c) = w2;
}

// Bidirectional attention.  Workgroup: 128 queries (wave w: queries 32 w .. 32 w + 31
// of the group, two 16-query tiles) of head h; keys in tiles of 64, double-buffered
// in LDS: each thread's share of the next tile is loaded into registers while the
// current tile is consumed and stored after it, so one barrier per tile suffices.
// Per key tile: S^T = K Q^T for both query tiles (8 MFMAs each), the tile's score
// maxima, then per query tile the probabilities and O^T += V^T P^T (8 MFMAs) with P^T
// taken straight from the S^T accumulators, and the probability sums by one more MFMA
// per 32 keys with an all-ones left operand: every lane then holds its query's sum
// (no cross-lane reduction), and the sums cover exactly the rounded probabilities
// that enter the product.  The running max (base 2, scaled) moves only when a tile's
// max exceeds it by more than 8, so probabilities stay below 2^8 (exact in the
// normalised result; fp32 sums) and the rescaling of the accumulators is rare.  Only
// the last key tile is masked.
__global__ __launch_bounds__(256) void sel_attention_kernel(const uint16_t* qk, const uint16_t* vt, int vt_pitch,
                                                            uint16_t* out, int T, int key_len, float* part) {
  constexpr int KT = 64;
  __shared__ uint16_t ks[2][KT][kDh + 8];  // key rows of the tile
  __shared__ uint16_t vs[2][kDh][KT + 8];  // value columns (channel-major) of the tile
  const int tid = threadIdx.x, lane = tid & 63, i16 = lane & 15, kg = lane >> 4, wv = tid >> 6;
  const int h = blockIdx.y;
  const int q_base = blockIdx.x * 128 + 32 * wv;
  const int kb = blockIdx.z * key_len, ke = min(T, kb + key_len);  // this workgroup's keys
  const float sc = 0.125f * kLog2e;  // 1/sqrt(64), base 2
  // the query operand (B of S^T = K Q^T): lane (query i16, kg) holds channels 8 kg .. + 7 of each k-step
  bf16x8 qb[2][2];
#pragma unroll
  for (int qt = 0; qt < 2; ++qt) {
    const int q = q_base + 16 * qt + i16;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      if (q < T) qb[qt][j] = *reinterpret_cast<const bf16x8*>(qk + (int64_t)q * (2 * kW) + h * kDh + 32 * j + 8 * kg);
      else qb[qt][j] = bf16x8{};
    }
  }
  // Staging share of a thread: 8 bf16 of key row (tid >> 3) + 32 hh and 8 keys of
  // value channel (tid >> 3) + 32 hh, both at offset 8 (tid & 7).
  const int sr = tid >> 3, s8 = 8 * (tid & 7);
  uint4 kreg[2], vreg[2];
  // whole tile inside the prompt: no checks
  auto fetch_full = [&](int k0) {
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      kreg[hh] = *reinterpret_cast<const uint4*>(qk + (int64_t)(k0 + sr + 32 * hh) * (2 * kW) + kW + h * kDh + s8);
      vreg[hh] = *reinterpret_cast<const uint4*>(vt + (int64_t)(h * kDh + sr + 32 * hh) * vt_pitch + k0 + s8);
    }
  };
  auto fetch = [&](int k0) {
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const int key = k0 + sr + 32 * hh;
      kreg[hh] = key < ke ? *reinterpret_cast<const uint4*>(qk + (int64_t)key * (2 * kW) + kW + h * kDh + s8)
                         : make_uint4(0, 0, 0, 0);
      const uint16_t* vp = vt + (int64_t)(h * kDh + sr + 32 * hh) * vt_pitch + k0 + s8;
      if (k0 + s8 + 8 <= ke) {
        vreg[hh] = *reinterpret_cast<const uint4*>(vp);
      } else {  // past the key range: zeros (their probabilities are 0, and 0 * garbage could be NaN)
        uint32_t w4[4];
        for (int e = 0; e < 4; ++e) {
          const uint32_t a0 = k0 + s8 + 2 * e < ke ? vp[2 * e] : 0u;
          const uint32_t a1 = k0 + s8 + 2 * e + 1 < ke ? vp[2 * e + 1] : 0u;
          w4[e] = a0 | (a1 << 16);
        }
        vreg[hh] = make_uint4(w4[0], w4[1], w4[2], w4[3]);
      }
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      *reinterpret_cast<uint4*>(&ks[buf][sr + 32 * hh][s8]) = kreg[hh];
      *reinterpret_cast<uint4*>(&vs[buf][sr + 32 * hh][s8]) = vreg[hh];
    }
  };
  bf16x8 ones;
#pragma unroll
  for (int e = 0; e < 8; ++e) ones[e] = (__bf16)1.0f;
  f4 o[2][4] = {}, lsum[2] = {};
  float m[2] = {-INFINITY, -INFINITY};
  auto tile = [&](int k0, int buf, auto last_tag) {
    constexpr bool kLast = decltype(last_tag)::value;
    // S^T tile tau (keys 16 tau .. + 15 of the tile): A = key rows; V^T operands of
    // the halves: lane (channel i16, kg) holds the keys of its k-slots, 4 kg .. + 3
    // and 16 + 4 kg .. + 3 of the half (the S^T accumulator order).
    bf16x8 ka[4][2], va[2][4];
#pragma unroll
    for (int tau = 0; tau < 4; ++tau)
#pragma unroll
      for (int j = 0; j < 2; ++j) ka[tau][j] = *reinterpret_cast<const bf16x8*>(&ks[buf][16 * tau + i16][32 * j + 8 * kg]);
#pragma unroll
    for (int hf = 0; hf < 2; ++hf)
#pragma unroll
      for (int ct = 0; ct < 4; ++ct) {
        const uint16_t* vr = &vs[buf][16 * ct + i16][32 * hf];
        const uint2 lo = *reinterpret_cast<const uint2*>(vr + 4 * kg);
        const uint2 hi = *reinterpret_cast<const uint2*>(vr + 16 + 4 * kg);
        va[hf][ct] = bitcast<bf16x8>(make_uint4(lo.x, lo.y, hi.x, hi.y));
      }
    // lane (query i16, kg) of s[qt][tau] holds the raw score of key 16 tau + 4 kg + e
    f4 s[2][4] = {};
#pragma unroll
    for (int qt = 0; qt < 2; ++qt)
#pragma unroll
      for (int tau = 0; tau < 4; ++tau)
#pragma unroll
        for (int j = 0; j < 2; ++j) s[qt][tau] = mfma_bf(ka[tau][j], qb[qt][j], s[qt][tau]);
    float mt[2];
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
      if constexpr (kLast) {  // mask the keys past the prompt
#pragma unroll
        for (int tau = 0; tau < 4; ++tau)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (k0 + 16 * tau + 4 * kg + e >= ke) s[qt][tau][e] = -INFINITY;
      }
      float mx = s[qt][0][0];
#pragma unroll
      for (int tau = 0; tau < 4; ++tau)
#pragma unroll
        for (int e = 0; e < 4; ++e) mx = fmaxf(mx, s[qt][tau][e]);
      mt[qt] = rows_max(mx) * sc;  // the scale enters the exponent
    }
    // move the running max (and rescale) only past a margin of 8; finite: the tile holds a key
    if (__builtin_amdgcn_ballot_w64(mt[0] > m[0] + 8.0f || mt[1] > m[1] + 8.0f)) {
#pragma unroll
      for (int qt = 0; qt < 2; ++qt) {
        const float mnew = fmaxf(m[qt], mt[qt]);
        const float alpha = __builtin_amdgcn_exp2f(m[qt] - mnew);
        m[qt] = mnew;
#pragma unroll
        for (int ct = 0; ct < 4; ++ct) o[qt][ct] *= alpha;
        lsum[qt] *= alpha;
      }
    }
    
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
      bf16x8 pb[2];
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
#pragma unroll
        for (int e = 0; e < 8; ++e)
          pb[hf][e] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(s[qt][2 * hf + (e >> 2)][e & 3], sc, -m[qt]));  // <= 2^8
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
#pragma unroll
        for (int ct = 0; ct < 4; ++ct) o[qt][ct] = mfma_bf(va[hf][ct], pb[hf], o[qt][ct]);
        lsum[qt] = mfma_bf(ones, pb[hf], lsum[qt]);
      }
    }
  };
  fetch(kb);
  stash(0);
  __syncthreads();
  int buf = 0, k0 = kb;
  for (; k0 + KT < ke; k0 += KT, buf ^= 1) {
    if (k0 + 2 * KT <= ke) fetch_full(k0 + KT);  // uniform
    else fetch(k0 + KT);
    tile(k0, buf, std::false_type{});
    stash(buf ^ 1);  // that buffer was last read before the previous barrier
    __syncthreads();
  }
  tile(k0, buf, std::true_type{});
  // O^T tiles: lane (query i16, kg) holds channels 16 ct + 4 kg + e
#pragma unroll
  for (int qt = 0; qt < 2; ++qt) {
    const int q = q_base + 16 * qt + i16;
    if (q >= T) continue;
    if (part) {  // a key split: unnormalised output, running max and sum for the merge
      float* rec = part + (((int64_t)blockIdx.z * T + q) * kHeads + h) * kRec;
#pragma unroll
      for (int ct = 0; ct < 4; ++ct) *reinterpret_cast<f4*>(rec + 16 * ct + 4 * kg) = o[qt][ct];
      if (kg == 0) {
        rec[kDh] = m[qt];
        rec[kDh + 1] = lsum[qt][0];
      }
      continue;
    }
    const float inv = 1.0f / lsum[qt][0];
#pragma unroll
    for (int ct = 0; ct < 4; ++ct)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        out[(int64_t)q * kW + h * kDh + 16 * ct + 4 * kg + e] = f32_to_bf16_bits(o[qt][ct][e] * inv);
  }
}

// Merge of the key splits: per (query, head), the splits' outputs weighted by
// 2^(m_s - M) over the merged sum.  One thread per 4 channels.
__global__ __launch_bounds__(256) void sel_attn_merge_kernel(const float* part, int splits, int T, uint16_t* out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)T * kHeads * (kDh / 4)) return;
  const int c4 = (int)(i % (kDh / 4));
  const int64_t qh = i / (kDh / 4);  // q * kHeads + h
  const int64_t stride = (int64_t)T * kHeads * kRec;
  const float* rec = part + qh * kRec;
  float M = rec[kDh];
  for (int sp = 1; sp < splits; ++sp) M = fmaxf(M, rec[sp * stride + kDh]);
  f4 acc = {0.f, 0.f, 0.f, 0.f};
  float L = 0.0f;
  for (int sp = 0; sp < splits; ++sp) {
    const float w = __builtin_amdgcn_exp2f(rec[sp * stride + kDh] - M);
    acc += w * *reinterpret_cast<const f4*>(rec + sp * stride + 4 * c4);
    L += w * rec[sp * stride + kDh + 1];
  }
  const float inv = 1.0f / L;
  uint2 w2;
  w2.x = (uint32_t)f32_to_bf16_bits(acc[0] * inv) | ((uint32_t)f32_to_bf16_bits(acc[1] * inv) << 16);
  w2.y = (uint32_t)f32_to_bf16_bits(acc[2] * inv) | ((uint32_t)f32_to_bf16_bits(acc[3] * inv) << 16);
  const int64_t q = qh / kHeads, h = qh % kHeads;
  *reinterpret_cast<uint2*>(out + q * kW + h * kDh + 4 * c4) = w2;
}

// Partial column sums of the RMS-normalised rows over chunks of 256 rows:
// part[chunk][c] = sum_t x[t][c] / rms(x[t]) (the final gain is applied to the
// mean).  Wave rg takes every fourth row of the chunk, lane c4 columns 4 c4 .. + 3;
// the four waves meet in LDS.
__global__ __launch_bounds__(256) void sel_pool_kernel(const float* x, float* part, int T) {
  __shared__ float red[4][kW];
  const int tid = threadIdx.x, c4 = tid & 63, rg = tid >> 6, chunk = blockIdx.x;
  const int t0 = chunk * 256, t1 = min(T, t0 + 256);
  f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
  for (int t = t0 + rg; t < t1; t += 4) {
    const f4 v = *reinterpret_cast<const f4*>(x + (int64_t)t * kW + 4 * c4);
    const float ms = wave_sum(v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3]) * (1.0f / kW);
    acc += v * (1.0f / sqrtf(ms + kRmsEps));
  }
  *reinterpret_cast<f4*>(&red[rg][4 * c4]) = acc;
  __syncthreads();
  part[(int64_t)chunk * kW + tid] = red[0][tid] + red[1][tid] + red[2][tid] + red[3][tid];
}

// One workgroup per layer l: the feature (thread c: the mean over the partial sums of
// channel c times the final gain, then the budget scale and shift), the layer's
// logits (products reduced over the 256 channels), and the argmax (the lowest
// action on ties; the depth action, index 0, never at layer 0 nor without depth).
__global__ __launch_bounds__(256) void sel_heads_kernel(const float* part, int n_chunks, int T, const uint16_t* g_final,
                                                        const float* film, const uint16_t* w_head,
                                                        const uint16_t* b_head, int n_actions, int depth,
                                                        float* logits, int32_t* action) {
  __shared__ float red[4][kMaxActions];
  const int c = threadIdx.x, lane = c & 63, wv = c >> 6, l = blockIdx.x;
  float f4s[4] = {0.0f, 0.0f, 0.0f, 0.0f};  // four independent chains over the chunks
  int k = 0;
  for (; k + 4 <= n_chunks; k += 4)
#pragma unroll
    for (int u = 0; u < 4; ++u) f4s[u] += part[(int64_t)(k + u) * kW + c];
  for (; k < n_chunks; ++k) f4s[0] += part[(int64_t)k * kW + c];
  float f = (f4s[0] + f4s[1] + f4s[2] + f4s[3]) / (float)T * bf16_to_f32(g_final[c]);
  if (film) f = fmaf(f, film[c], f) + film[kW + c];
  for (int a = 0; a < n_actions; ++a) {
    const float z = wave_sum(f * bf16_to_f32(w_head[((int64_t)l * n_actions + a) * kW + c]));
    if (lane == 0) red[wv][a] = z;
  }
  __syncthreads();
  if (c == 0) {
    int best = 0;
    float zb = -INFINITY;
    for (int a = 0; a < n_actions; ++a) {
      float v = red[0][a] + red[1][a] + red[2][a] + red[3][a] + bf16_to_f32(b_head[l * n_actions + a]);
      if (a == 0 && (l == 0 || !depth)) v = -INFINITY;
      if (logits) logits[l * n_actions + a] = v;
      if (a == 0 || v > zb) {
        best = a;
        zb = v;
      }
    }
    action[l] = best;
  }
}

// Packed weight offsets (bf16 elements).
struct SelOffsets {
  int64_t w_in, blk[2], g_final, w_head, b_head, total;
};
// per block: g_attn, w_qkv [768][256], w_o [256][256], g_ffn, w_gate|w_up [2048][256], w_down [256][1024]
constexpr int64_t kBlockElems = kW + (int64_t)3 * kW * kW + (int64_t)kW * kW + kW + (int64_t)2 * kFfn * kW +
                                (int64_t)kW * kFfn;

SelOffsets sel_offsets(int d_model, int L, int A) {
  SelOffsets o;
  o.w_in = 0;
  o.blk[0] = (int64_t)kW * d_model;
  o.blk[1] = o.blk[0] + kBlockElems;
  o.g_final = o.blk[1] + kBlockElems;
  o.w_head = o.g_final + kW;
  o.b_head = o.w_head + (int64_t)L * A * kW;
  o.total = o.b_head + (int64_t)L * A;
  return o;
}

struct SelWorkspace {
  int64_t x, h, qk, vt, f1, rope, part, splitk, attn, total;  // byte offsets
  int vt_pitch;
};

// Key splits of the attention when its 128-query workgroups alone would be fewer
// than about 512: each split at least 256 keys, a multiple of 64; no empty split.
// Returns the split count; *key_len gets the keys per split.
int sel_attn_splits(int T, int* key_len) {
  const int wgs = (T + 127) / 128 * kHeads;
  const int sp = std::min((512 + wgs - 1) / wgs, T / 256);
  if (sp <= 1) {
    *key_len = T;
    return 1;
  }
  *key_len = ((T + sp - 1) / sp + 63) / 64 * 64;
  return (T + *key_len - 1) / *key_len;
}

// Split-K for the long-K GEMMs with 256 output columns (the input map, K = d_model,
// and the down projection, K = 1024) when their 64-row tiles alone would give few
// workgroups: enough splits for about 512 workgroups, at most 16, each split at
// least 8 k-steps of 32.
constexpr int kSplitMax = 16;
int sel_splits(int T, int K) {
  const int row_blocks = (T + 63) / 64;
  int sp = std::min(std::min(kSplitMax, K / 256), (512 + row_blocks - 1) / row_blocks);
  if (sp <= 1) return 1;
  const int ksteps = K / 32, per = (ksteps + sp - 1) / sp;
  return (ksteps + per - 1) / per;  // no empty split
}

SelWorkspace sel_workspace(int T) {
  SelWorkspace w;
  const int Tp = (T + 31) / 32 * 32;
  w.vt_pitch = Tp;
  w.x = 0;                                                   // fp32 [T][256] residual stream
  w.h = kvk::round256(w.x + (int64_t)Tp * kW * 4);           // bf16 [T][256] normalised / attention output
  w.qk = kvk::round256(w.h + (int64_t)Tp * kW * 2);          // bf16 [T][512] rotated q | k
  w.vt = kvk::round256(w.qk + (int64_t)Tp * 2 * kW * 2);     // bf16 [256][Tp]
  w.f1 = kvk::round256(w.vt + (int64_t)kW * Tp * 2);         // bf16 [T][1024] SiLU(gate) * up
  w.rope = kvk::round256(w.f1 + (int64_t)Tp * kFfn * 2);     // fp32 [T][32] (cos, sin)
  w.part = kvk::round256(w.rope + (int64_t)Tp * (kDh / 2) * 8);  // fp32 [chunks][256]
  w.splitk = kvk::round256(w.part + (int64_t)((T + 255) / 256) * kW * 4);  // fp32 [splits][T][256]
  const int max_splits = std::min(kSplitMax, (512 + (T + 63) / 64 - 1) / ((T + 63) / 64));
  w.attn = kvk::round256(w.splitk + (max_splits > 1 ? (int64_t)max_splits * T * kW * 4 : 0));  // fp32 [splits][T][4][kRec]
  int key_len = 0;
  const int attn_splits = sel_attn_splits(T, &key_len);
  w.total = kvk::round256(w.attn + (attn_splits > 1 ? (int64_t)attn_splits * T * kHeads * kRec * 4 : 0));
  return w;
}

}  // namespace

using namespace kvk;

extern "C" kvk_status kvk_selector_workspace_bytes(int32_t d_model, int32_t n_layers, int32_t n_tokens,
                                                   size_t* out) {
  if (!out) return fail(KVK_ERR_INVALID, "selector: NULL output");
  if (d_model < 32 || d_model % 32 || n_layers < 1 || n_layers > KVK_MAX_LAYERS || n_tokens < 1)
    return fail(KVK_ERR_INVALID, "selector: d_model %d (multiple of 32), n_layers %d, n_tokens %d", d_model,
                n_layers, n_tokens);
  *out = (size_t)sel_workspace(n_tokens).total;
  return KVK_OK;
}

extern "C" int64_t kvk_selector_weight_elems(int32_t d_model, int32_t n_layers, int32_t n_actions) {
  if (d_model < 32 || d_model % 32 || n_layers < 1 || n_layers > KVK_MAX_LAYERS || n_actions < 2 ||
      n_actions > kMaxActions)
    return -1;
  return sel_offsets(d_model, n_layers, n_actions).total;
}

extern "C" kvk_status kvk_selector_forward(int32_t d_model, int32_t n_layers, int32_t n_actions, int32_t depth,
                                           const void* weights, const void* emb, int32_t n_tokens,
                                           const float* film, float* logits, int32_t* actions,
                                           void* workspace, size_t ws_bytes, hipStream_t stream) {
  size_t need = 0;
  kvk_status st = kvk_selector_workspace_bytes(d_model, n_layers, n_tokens, &need);
  if (st != KVK_OK) return st;
  if (n_actions < 2 || n_actions > kMaxActions)
    return fail(KVK_ERR_INVALID, "selector: n_actions %d outside 2..%d", n_actions, kMaxActions);
  if (depth != 0 && depth != 1) return fail(KVK_ERR_INVALID, "selector: depth flag %d (0 or 1)", depth);
  if (!weights || !emb || !actions || !workspace) return fail(KVK_ERR_INVALID, "selector: NULL buffer");
  if (need > ws_bytes) return fail(KVK_ERR_BUFFER, "selector: workspace %zu bytes < %zu needed", ws_bytes, need);
  if ((reinterpret_cast<uintptr_t>(weights) & 15) || (reinterpret_cast<uintptr_t>(emb) & 15) ||
      (reinterpret_cast<uintptr_t>(workspace) & 255) || (reinterpret_cast<uintptr_t>(logits) & 3) ||
      (reinterpret_cast<uintptr_t>(actions) & 3) || (reinterpret_cast<uintptr_t>(film) & 3))
    return fail(KVK_ERR_INVALID, "selector: misaligned buffer (weights/emb 16 B, workspace 256 B)");
  if (kvk_status st2 = check_gpu_buffers({weights, emb, film, logits, actions, workspace}, "kvk_selector_forward"))
    return st2;
  const SelOffsets O = sel_offsets(d_model, n_layers, n_actions);
  const SelWorkspace Wk = sel_workspace(n_tokens);
  const uint16_t* wp = static_cast<const uint16_t*>(weights);
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  float* x = reinterpret_cast<float*>(ws + Wk.x);
  uint16_t* hbuf = reinterpret_cast<uint16_t*>(ws + Wk.h);
  uint16_t* qk = reinterpret_cast<uint16_t*>(ws + Wk.qk);
  uint16_t* vt = reinterpret_cast<uint16_t*>(ws + Wk.vt);
  uint16_t* f1 = reinterpret_cast<uint16_t*>(ws + Wk.f1);
  float2* rope = reinterpret_cast<float2*>(ws + Wk.rope);
  float* part = reinterpret_cast<float*>(ws + Wk.part);
  const int T = n_tokens;
  auto gemm = [&](int epi, const uint16_t* a, int64_t w_off, int N, int K) {
    GemmArgs g;
    g.a = a;
    g.w = wp + w_off;
    g.out_f32 = x;
    g.out_bf16 = epi == kSwiGlu ? f1 : qk;
    g.vt = vt;
    g.rope = rope;
    g.M = T;
    g.N = N;
    g.K = K;
    g.vt_pitch = Wk.vt_pitch;
    const int splits = (epi == kStoreF32 || epi == kAddF32) ? sel_splits(T, K) : 1;
    g.k_len = (K / 32 + splits - 1) / splits * 32;
    g.part = splits > 1 ? reinterpret_cast<float*>(ws + Wk.splitk) : nullptr;
    const dim3 grid((unsigned)((T + 63) / 64), (unsigned)(N / 256), (unsigned)splits), blk(256);
    switch (epi) {
      case kStoreF32: hipLaunchKernelGGL(sel_gemm_kernel<kStoreF32>, grid, blk, 0, stream, g); break;
      case kAddF32: hipLaunchKernelGGL(sel_gemm_kernel<kAddF32>, grid, blk, 0, stream, g); break;
      case kSwiGlu: hipLaunchKernelGGL(sel_gemm_kernel<kSwiGlu>, grid, blk, 0, stream, g); break;
      default: hipLaunchKernelGGL(sel_gemm_kernel<kQkv>, grid, blk, 0, stream, g); break;
    }
    if (splits > 1) {
      const dim3 rgrid((unsigned)(((int64_t)T * (kW / 4) + 255) / 256));
      if (epi == kAddF32)
        hipLaunchKernelGGL(sel_splitk_kernel<kAddF32>, rgrid, blk, 0, stream, g.part, splits, x, T);
      else
        hipLaunchKernelGGL(sel_splitk_kernel<kStoreF32>, rgrid, blk, 0, stream, g.part, splits, x, T);
    }
  };
  const dim3 rows((unsigned)((T + 3) / 4)), b256(256);
  hipLaunchKernelGGL(sel_rope_kernel, dim3((unsigned)(((int64_t)T * (kDh / 2) + 255) / 256)), b256, 0, stream,
                     rope, T);
  gemm(kStoreF32, static_cast<const uint16_t*>(emb), O.w_in, kW, d_model);
  for (int bi = 0; bi < 2; ++bi) {
    const int64_t p = O.blk[bi];
    const int64_t g_attn = p, w_qkv = p + kW, w_o = w_qkv + (int64_t)3 * kW * kW, g_ffn = w_o + (int64_t)kW * kW,
                  w_gu = g_ffn + kW, w_down = w_gu + (int64_t)2 * kFfn * kW;
    hipLaunchKernelGGL(sel_rmsnorm_kernel, rows, b256, 0, stream, x, wp + g_attn, hbuf, T);
    gemm(kQkv, hbuf, w_qkv, 3 * kW, kW);
    {
      int key_len = 0;
      const int sp = sel_attn_splits(T, &key_len);
      float* apart = sp > 1 ? reinterpret_cast<float*>(ws + Wk.attn) : nullptr;
      hipLaunchKernelGGL(sel_attention_kernel, dim3((unsigned)((T + 127) / 128), kHeads, (unsigned)sp), b256, 0,
                         stream, qk, vt, Wk.vt_pitch, hbuf, T, key_len, apart);
      if (sp > 1)
        hipLaunchKernelGGL(sel_attn_merge_kernel, dim3((unsigned)(((int64_t)T * kHeads * (kDh / 4) + 255) / 256)),
                           b256, 0, stream, apart, sp, T, hbuf);
    }
    gemm(kAddF32, hbuf, w_o, kW, kW);
    hipLaunchKernelGGL(sel_rmsnorm_kernel, rows, b256, 0, stream, x, wp + g_ffn, hbuf, T);
    gemm(kSwiGlu, hbuf, w_gu, 2 * kFfn, kW);
    gemm(kAddF32, f1, w_down, kW, kFfn);
  }
  const int chunks = (T + 255) / 256;
  hipLaunchKernelGGL(sel_pool_kernel, dim3((unsigned)chunks), b256, 0, stream, x, part, T);
  hipLaunchKernelGGL(sel_heads_kernel, dim3((unsigned)n_layers), b256, 0, stream, part, chunks, T, wp + O.g_final,
                     film, wp + O.w_head, wp + O.b_head, n_actions, depth, logits, actions);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(KVK_ERR_DEVICE, "selector launch: %s", hipGetErrorString(e));
  return KVK_OK;
}
