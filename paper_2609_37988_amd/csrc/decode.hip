// Decode-step attention over per-layer compressed GQA caches (D1 + C1).
//
// KV-Kaizen §2.1: every layer attends with its own query over the keys and values
// of its anchor (itself, or the nearest earlier producing layer).  Layers that
// share an anchor are served together: their query rows are stacked so that the
// anchor's bytes are read once per step.  Decode is bound by reading the cache
// (§1), so the kernel streams each (sequence, KV head) stream once, split along
// the context into pieces of about 256 KiB; a second kernel merges the splits by
// log-sum-exp.
//
// Work unit: one 64-lane wave per (anchor item, sequence, KV head, split).  The
// query rows of the unit (G query heads x the layers that read the anchor, up to
// 16 per "chunk", up to 4 chunks) are the N = 16 columns of MFMA tiles:
//   S^T[token, row] = K_hat[token, :] . q[row, :]      (v_mfma_f32_16x16x32_{f16,bf16})
//   O^T[chan,  row] += V_hat^T[chan, token] . P^T[token, row]
// so every per-row quantity (running max, sum, rescale factor) lives in lane
// (lane % 16) and needs no transposition.  The block layout of include/kvk.h puts
// each lane's MFMA operands in contiguous bytes.
//
// Precision: integer codes are exact in fp16.  KIVI32 keys carry a scale and zero
// per (channel, 32 tokens); the scale is folded into the query once per block
// (q' = q * s, split into fp16 hi + lo so that q' keeps ~22 bits) and the zero
// enters as a per-row constant sum_c q_c z_c.  Values are dequantised to fp16
// (one rounding) and the probabilities enter as fp16.  bf16 blocks use bf16 MFMA
// with the query and probabilities split into bf16 hi + lo.  All accumulation is
// fp32.
#include <hip/hip_runtime.h>

#include "kvk_device.h"
#include "kvk_internal.h"

using namespace kvkd;

namespace {

constexpr int kMaxItems = KVK_MAX_LAYERS;
constexpr float kLog2e = 1.4426950408889634f;

struct DecodeItem {
  int64_t region;        // byte offset of the anchor's region in the arena
  int32_t stream_bytes;
  int32_t block_bytes;
  int32_t bits;
  int32_t q_layer0;      // first reading layer, relative to layer_begin
  int32_t geff;          // query rows: G * readers
  int32_t nsplit;
  int32_t split_blocks;
  int32_t wave_begin;    // first wave of this item within the launch (a multiple of 4)
  int32_t ws_off;        // float offset of the item's partials
  int32_t nchp;          // waves per (stream, split): 16-row chunks, padded to 1, 2 or 4
};

struct DecodeArgs {
  const uint8_t* arena;
  const void* q;
  float* ws;
  int32_t q_f32;
  int32_t B, Hq, Hkv, G;
  int32_t nbf;       // full blocks stored per stream
  int32_t ntail;     // tokens in the tail block
  int32_t nb_cap;
  int32_t total_waves;
  int32_t n_items;
  float scale_log2;  // softmax scale * log2(e)
  DecodeItem items[kMaxItems];
};

struct CombineArgs {
  float* out;
  const float* ws;
  int32_t B, Hq, Hkv, G;
  int32_t n_rows;  // layers * B * Hq
  int32_t n_layers;
  int32_t layer_item[kMaxItems];
  int32_t layer_slot0[kMaxItems];
  int32_t item_ws_off[kMaxItems];
  int32_t item_nsplit[kMaxItems];
  int32_t item_geff[kMaxItems];
};

__device__ __forceinline__ f4 mfma16(half8 a, half8 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f4 mfmab(bf16x8 a, bf16x8 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float wave_max_kg(float x) {
  x = fmaxf(x, __shfl_xor(x, 16));
  x = fmaxf(x, __shfl_xor(x, 32));
  return x;
}
__device__ __forceinline__ float wave_sum_kg(float x) {
  x += __shfl_xor(x, 16);
  x += __shfl_xor(x, 32);
  return x;
}

__device__ __forceinline__ bf16x8 to_bf16x8(const float* x) {
  bf16x8 r;
#pragma unroll
  for (int s = 0; s < 8; ++s) r[s] = (__bf16)x[s];
  return r;
}

// Per-wave state of one work unit.
template <int D, int NCH>
struct Unit {
  static constexpr int NJ = D / 32;  // K sub-chunks (MFMA k-steps over channels)
  static constexpr int NM = D / 16;  // V channel tiles
  float q[NCH][NJ][8];               // query rows, fp32, lane's channels
  f4 o[NCH][NM];                     // output accumulators (O^T tiles)
  float m[NCH];                      // running max (log2 domain), per row
  float l[NCH];                      // lane-partial running sum
};

// Online-softmax update from the 8 logits of a 32-token block (2 tiles x 4),
// returning the probabilities in place.
template <int D, int NCH>
__device__ __forceinline__ void softmax_update(Unit<D, NCH>& u, float (&x)[NCH][8]) {
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    float mb = x[c][0];
#pragma unroll
    for (int e = 1; e < 8; ++e) mb = fmaxf(mb, x[c][e]);
    mb = wave_max_kg(mb);
    const float mnew = fmaxf(u.m[c], mb);
    const float alpha = (u.m[c] == -INFINITY) ? 0.0f : exp2f(u.m[c] - mnew);
    float ps = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float p = (x[c][e] == -INFINITY) ? 0.0f : exp2f(x[c][e] - mnew);
      x[c][e] = p;
      ps += p;
    }
    u.l[c] = u.l[c] * alpha + ps;
    u.m[c] = mnew;
    if (__any(alpha != 1.0f)) {
#pragma unroll
      for (int mt = 0; mt < Unit<D, NCH>::NM; ++mt) u.o[c][mt] *= alpha;
    }
  }
}

// The query rows as bf16 hi + lo pairs (for bf16 blocks).
template <int D, int NCH>
struct QB16 {
  bf16x8 hi[NCH][D / 32], lo[NCH][D / 32];
};

template <int D, int NCH>
__device__ __forceinline__ void make_qb16(const Unit<D, NCH>& u, QB16<D, NCH>& qb) {
#pragma unroll
  for (int c = 0; c < NCH; ++c)
#pragma unroll
    for (int j = 0; j < D / 32; ++j) {
      float hi[8], lo[8];
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        hi[s] = (float)(__bf16)u.q[c][j][s];
        lo[s] = u.q[c][j][s] - hi[s];
      }
      qb.hi[c][j] = to_bf16x8(hi);
      qb.lo[c][j] = to_bf16x8(lo);
    }
}

// A bf16 block (a b = 16 layer's block, or any layer's tail) with `nvalid` tokens.
template <int D, int NCH>
__device__ __forceinline__ void block_bf16(Unit<D, NCH>& u, const QB16<D, NCH>& qb, const uint8_t* blk,
                                           int lane, int nvalid, float sl2) {
  constexpr int NJ = D / 32, NM = D / 16;
  const int kg = lane >> 4;
  float x[NCH][8];
#pragma unroll
  for (int tau = 0; tau < 2; ++tau) {
    const uint4* kp = reinterpret_cast<const uint4*>(blk + 32 * D * tau + lane * (D / 2));
    bf16x8 kop[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j) kop[j] = bitcast<bf16x8>(kp[j]);
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        acc = mfmab(kop[j], qb.hi[c][j], acc);
        acc = mfmab(kop[j], qb.lo[c][j], acc);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int tok = 16 * tau + 4 * kg + r;
        x[c][4 * tau + r] = tok < nvalid ? acc[r] * sl2 : -INFINITY;
      }
    }
  }
  softmax_update<D, NCH>(u, x);
  bf16x8 phi[NCH], plo[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    float h[8], lw[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      h[e] = (float)(__bf16)x[c][e];
      lw[e] = x[c][e] - h[e];
    }
    phi[c] = to_bf16x8(h);
    plo[c] = to_bf16x8(lw);
  }
  const uint4* vp = reinterpret_cast<const uint4*>(blk + 64 * D + lane * D);
#pragma unroll
  for (int mt = 0; mt < NM; ++mt) {
    const bf16x8 vop = bitcast<bf16x8>(vp[mt]);
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      u.o[c][mt] = mfmab(vop, phi[c], u.o[c][mt]);
      u.o[c][mt] = mfmab(vop, plo[c], u.o[c][mt]);
    }
  }
}

// Load the lane's K code chunks of tile tau and unpack them to exact fp16 (minus off).
template <int D, int BITS>
__device__ __forceinline__ void load_k_codes(const uint8_t* blk, int tau, int lane, float off,
                                             half8 (&kop)[D / 32]) {
  constexpr int NJ = D / 32;
  const uint8_t* p = blk + 2 * D * BITS * tau + lane * (D * BITS / 32);
  if constexpr (BITS == 4) {
    const uint32_t* w = reinterpret_cast<const uint32_t*>(p);
    uint32_t wr[NJ];
    if constexpr (NJ == 4) {
      const uint4 v = *reinterpret_cast<const uint4*>(p);
      wr[0] = v.x; wr[1] = v.y; wr[2] = v.z; wr[3] = v.w;
    } else {
#pragma unroll
      for (int j = 0; j < NJ; ++j) wr[j] = w[j];
    }
#pragma unroll
    for (int j = 0; j < NJ; ++j) kop[j] = unpack4(wr[j], off);
  } else if constexpr (BITS == 8) {
    const uint4* w = reinterpret_cast<const uint4*>(p);
#pragma unroll
    for (int j2 = 0; j2 < NJ / 2; ++j2) {
      const uint4 v = w[j2];
      kop[2 * j2] = unpack8(v.x, v.y, off);
      kop[2 * j2 + 1] = unpack8(v.z, v.w, off);
    }
  } else {  // BITS == 2
    const uint32_t* w = reinterpret_cast<const uint32_t*>(p);
#pragma unroll
    for (int j2 = 0; j2 < NJ / 2; ++j2) unpack2(w[j2], off, kop[2 * j2], kop[2 * j2 + 1]);
  }
}

// Load the lane's V code chunks (all channel tiles) as exact fp16 (minus off).
template <int D, int BITS>
__device__ __forceinline__ void load_v_codes(const uint8_t* blk, int lane, float off,
                                             half8 (&vop)[D / 16]) {
  constexpr int NM = D / 16;
  const uint8_t* p = blk + 4 * D * BITS + lane * (D * BITS / 16);
  if constexpr (BITS == 4) {
    const uint4* w = reinterpret_cast<const uint4*>(p);
#pragma unroll
    for (int m4 = 0; m4 < NM / 4; ++m4) {
      const uint4 v = w[m4];
      vop[4 * m4 + 0] = unpack4(v.x, off);
      vop[4 * m4 + 1] = unpack4(v.y, off);
      vop[4 * m4 + 2] = unpack4(v.z, off);
      vop[4 * m4 + 3] = unpack4(v.w, off);
    }
  } else if constexpr (BITS == 8) {
    const uint4* w = reinterpret_cast<const uint4*>(p);
#pragma unroll
    for (int m2 = 0; m2 < NM / 2; ++m2) {
      const uint4 v = w[m2];
      vop[2 * m2] = unpack8(v.x, v.y, off);
      vop[2 * m2 + 1] = unpack8(v.z, v.w, off);
    }
  } else {
    const uint32_t* w = reinterpret_cast<const uint32_t*>(p);
#pragma unroll
    for (int m2 = 0; m2 < NM / 2; ++m2) unpack2(w[m2], off, vop[2 * m2], vop[2 * m2 + 1]);
  }
}

// A full KIVI32 block of `BITS`-bit codes.
template <int D, int NCH, int BITS>
__device__ __forceinline__ void block_kivi(Unit<D, NCH>& u, const uint8_t* blk, int lane, float sl2) {
  constexpr int NJ = D / 32, NM = D / 16;
  const int kg = lane >> 4;
  const _Float16* kmeta = reinterpret_cast<const _Float16*>(blk + 8 * D * BITS);
  const _Float16* vmeta = kmeta + 2 * D;
  // q' = q * s (hi + lo in fp16) and the zero term sum_c q_c z_c, per row.
  half8 qh[NCH][NJ], ql[NCH][NJ];
  float zt[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c) zt[c] = 0.0f;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const half8 sv = *reinterpret_cast<const half8*>(kmeta + 32 * j + 8 * kg);
    const half8 zv = *reinterpret_cast<const half8*>(kmeta + D + 32 * j + 8 * kg);
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const float qs = u.q[c][j][s] * (float)sv[s];
        const _Float16 h = (_Float16)qs;
        qh[c][j][s] = h;
        ql[c][j][s] = (_Float16)(qs - (float)h);
        zt[c] = fmaf(u.q[c][j][s], (float)zv[s], zt[c]);
      }
    }
  }
#pragma unroll
  for (int c = 0; c < NCH; ++c) zt[c] = wave_sum_kg(zt[c]);

  float x[NCH][8];
#pragma unroll
  for (int tau = 0; tau < 2; ++tau) {
    half8 kop[NJ];
    load_k_codes<D, BITS>(blk, tau, lane, 0.0f, kop);
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        acc = mfma16(kop[j], qh[c][j], acc);
        acc = mfma16(kop[j], ql[c][j], acc);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) x[c][4 * tau + r] = (acc[r] + zt[c]) * sl2;
    }
  }
  softmax_update<D, NCH>(u, x);
  half8 p[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c)
#pragma unroll
    for (int e = 0; e < 8; ++e) p[c][e] = (_Float16)x[c][e];

  half8 vop[NM];
  load_v_codes<D, BITS>(blk, lane, 0.0f, vop);
#pragma unroll
  for (int g = 0; g < D / 32; ++g) {
    const half8 vs = *reinterpret_cast<const half8*>(vmeta + ((g * 2 + 0) * 4 + kg) * 8);
    const half8 vz = *reinterpret_cast<const half8*>(vmeta + ((g * 2 + 1) * 4 + kg) * 8);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int mt = 2 * g + h;
      const half8 vh = __builtin_elementwise_fma(vop[mt], vs, vz);  // fp16 dequantised values
#pragma unroll
      for (int c = 0; c < NCH; ++c) u.o[c][mt] = mfma16(vh, p[c], u.o[c][mt]);
    }
  }
}

// A full SYMROW block: per-token scales factor out of both contractions.
template <int D, int NCH, int BITS>
__device__ __forceinline__ void block_symrow(Unit<D, NCH>& u, const half8 (&qh)[NCH][D / 32],
                                             const half8 (&ql)[NCH][D / 32], const uint8_t* blk,
                                             int lane, float sl2) {
  constexpr int NJ = D / 32, NM = D / 16;
  const int kg = lane >> 4;
  const float off = (float)(1 << (BITS - 1));
  const uint16_t* ksc = reinterpret_cast<const uint16_t*>(blk + 8 * D * BITS);
  const uint16_t* vsc = ksc + 32;
  float x[NCH][8];
#pragma unroll
  for (int tau = 0; tau < 2; ++tau) {
    half8 kop[NJ];
    load_k_codes<D, BITS>(blk, tau, lane, off, kop);
    float sk[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) sk[r] = bf16_to_f32(ksc[16 * tau + 4 * kg + r]) * sl2;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        acc = mfma16(kop[j], qh[c][j], acc);
        acc = mfma16(kop[j], ql[c][j], acc);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) x[c][4 * tau + r] = acc[r] * sk[r];
    }
  }
  softmax_update<D, NCH>(u, x);
  float sv[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) sv[e] = bf16_to_f32(vsc[16 * (e >> 2) + 4 * kg + (e & 3)]);
  half8 p[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c)
#pragma unroll
    for (int e = 0; e < 8; ++e) p[c][e] = (_Float16)(x[c][e] * sv[e]);
  half8 vop[NM];
  load_v_codes<D, BITS>(blk, lane, off, vop);
#pragma unroll
  for (int mt = 0; mt < NM; ++mt)
#pragma unroll
    for (int c = 0; c < NCH; ++c) u.o[c][mt] = mfma16(vop[mt], p[c], u.o[c][mt]);
}

template <int D, int NCH, int BITS, bool KIVI>
__device__ __forceinline__ void run_stream(Unit<D, NCH>& u, const uint8_t* stream, const DecodeArgs& a,
                                           const DecodeItem& it, int k0, int k1, int lane) {
  constexpr int NJ = D / 32;
  const float sl2 = a.scale_log2;
  half8 qh[NCH][NJ], ql[NCH][NJ];
  if constexpr (!KIVI && BITS != 16) {
#pragma unroll
    for (int c = 0; c < NCH; ++c)
#pragma unroll
      for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int s = 0; s < 8; ++s) {
          const _Float16 h = (_Float16)u.q[c][j][s];
          qh[c][j][s] = h;
          ql[c][j][s] = (_Float16)(u.q[c][j][s] - (float)h);
        }
  }
  QB16<D, NCH> qb;
  if constexpr (BITS == 16) make_qb16<D, NCH>(u, qb);
  const int kfull = min(k1, a.nbf);
  for (int k = k0; k < kfull; ++k) {
    const uint8_t* blk = stream + (int64_t)k * it.block_bytes;
    if constexpr (BITS == 16) {
      block_bf16<D, NCH>(u, qb, blk, lane, 32, sl2);
    } else if constexpr (KIVI) {
      block_kivi<D, NCH, BITS>(u, blk, lane, sl2);
    } else {
      block_symrow<D, NCH, BITS>(u, qh, ql, blk, lane, sl2);
    }
  }
  if (k1 > a.nbf) {  // this split holds the tail block
    if constexpr (BITS != 16) make_qb16<D, NCH>(u, qb);
    block_bf16<D, NCH>(u, qb, stream + (int64_t)a.nb_cap * it.block_bytes, lane, a.ntail, sl2);
  }
}

template <int D, bool KIVI>
__global__ __launch_bounds__(256) void gqa_decode_kernel(DecodeArgs a) {
  constexpr int NJ = D / 32, NM = D / 16;
  const int lane = threadIdx.x & 63;
  const int wave = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (wave >= a.total_waves) return;
  int ii = 0;
  while (ii + 1 < a.n_items && a.items[ii + 1].wave_begin <= wave) ++ii;
  const DecodeItem& it = a.items[ii];
  const int local = wave - it.wave_begin;
  const int chunk = local % it.nchp;
  const int unit = local / it.nchp;
  if (unit >= a.B * a.Hkv * it.nsplit || 16 * chunk >= it.geff) return;  // alignment padding
  const int split = unit % it.nsplit;
  const int sidx = unit / it.nsplit;  // b * Hkv + kvh
  const int b = sidx / a.Hkv, kvh = sidx % a.Hkv;
  const int i16 = lane & 15, kg = lane >> 4;
  const int row = 16 * chunk + i16;  // query row of this lane: (reader layer, head in group)

  Unit<D, 1> u;
  u.m[0] = -INFINITY;
  u.l[0] = 0.0f;
#pragma unroll
  for (int mt = 0; mt < NM; ++mt) u.o[0][mt] = f4{0.f, 0.f, 0.f, 0.f};
  {
    const bool valid = row < it.geff;
    const int r = row / a.G, gh = row % a.G;
    const int64_t qrow = (((int64_t)(it.q_layer0 + r) * a.B + b) * a.Hq + kvh * a.G + gh) * D;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int ch = 32 * j + 8 * kg;
      if (!valid) {
#pragma unroll
        for (int s = 0; s < 8; ++s) u.q[0][j][s] = 0.0f;
      } else if (a.q_f32) {
        const float4* qp = reinterpret_cast<const float4*>(static_cast<const float*>(a.q) + qrow + ch);
        const float4 v0 = qp[0], v1 = qp[1];
        u.q[0][j][0] = v0.x; u.q[0][j][1] = v0.y; u.q[0][j][2] = v0.z; u.q[0][j][3] = v0.w;
        u.q[0][j][4] = v1.x; u.q[0][j][5] = v1.y; u.q[0][j][6] = v1.z; u.q[0][j][7] = v1.w;
      } else {
        const uint4 v = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(a.q) + qrow + ch);
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          u.q[0][j][2 * p] = __uint_as_float(w[p] << 16);
          u.q[0][j][2 * p + 1] = __uint_as_float(w[p] & 0xffff0000u);
        }
      }
    }
  }

  const int nblk = a.nbf + (a.ntail > 0 ? 1 : 0);
  const int k0 = split * it.split_blocks;
  const int k1 = min(nblk, k0 + it.split_blocks);
  const uint8_t* stream = a.arena + it.region + (int64_t)sidx * it.stream_bytes;
  switch (it.bits) {
    case 16: run_stream<D, 1, 16, KIVI>(u, stream, a, it, k0, k1, lane); break;
    case 8: run_stream<D, 1, 8, KIVI>(u, stream, a, it, k0, k1, lane); break;
    case 4: run_stream<D, 1, 4, KIVI>(u, stream, a, it, k0, k1, lane); break;
    default: run_stream<D, 1, 2, KIVI>(u, stream, a, it, k0, k1, lane); break;
  }

  // partials: rows of (o[D], m, l, pad, pad)
  float* base = a.ws + it.ws_off + ((int64_t)sidx * it.nsplit + split) * it.geff * (D + 4);
  const float lt = wave_sum_kg(u.l[0]);
  if (row < it.geff) {
    float* pr = base + (int64_t)row * (D + 4);
#pragma unroll
    for (int mt = 0; mt < NM; ++mt) *reinterpret_cast<f4*>(pr + 16 * mt + 4 * kg) = u.o[0][mt];
    if (kg == 0) {
      pr[D] = u.m[0];
      pr[D + 1] = lt;
    }
  }
}

// Merge the splits of every output row by log-sum-exp: one wave per (layer, b, head).
template <int D>
__global__ __launch_bounds__(256) void gqa_combine_kernel(CombineArgs a) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= a.n_rows) return;
  const int li = row / (a.B * a.Hq);
  const int rem = row % (a.B * a.Hq);
  const int b = rem / a.Hq, h = rem % a.Hq;
  const int item = a.layer_item[li];
  const int slot = a.layer_slot0[li] + h % a.G;
  const int kvh = h / a.G;
  const int nsplit = a.item_nsplit[item], geff = a.item_geff[item];
  const float* base = a.ws + a.item_ws_off[item] +
                      (((int64_t)(b * a.Hkv + kvh) * nsplit) * geff + slot) * (D + 4);
  const int64_t stride = (int64_t)geff * (D + 4);
  float mstar = -INFINITY;
  for (int s = lane; s < nsplit; s += 64) mstar = fmaxf(mstar, base[s * stride + D]);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) mstar = fmaxf(mstar, __shfl_xor(mstar, off));
  float lsum = 0.0f;
  constexpr int PER = D / 64;
  float acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) acc[e] = 0.0f;
  for (int s = 0; s < nsplit; ++s) {
    const float* p = base + s * stride;
    const float ms = p[D];
    const float w = (ms == -INFINITY) ? 0.0f : exp2f(ms - mstar);
    lsum = fmaf(w, p[D + 1], lsum);
#pragma unroll
    for (int e = 0; e < PER; ++e) acc[e] = fmaf(w, p[lane + 64 * e], acc[e]);
  }
  const float inv = lsum > 0.0f ? 1.0f / lsum : 0.0f;
  float* o = a.out + (int64_t)row * D;
#pragma unroll
  for (int e = 0; e < PER; ++e) o[lane + 64 * e] = acc[e] * inv;
}

}  // namespace

using namespace kvk;

namespace {

// Everything one decode call launches: the D1 arguments (all anchors of the
// range in one launch) and the C1 arguments.
struct DecodePlan {
  DecodeArgs d1;
  CombineArgs c1;
  int kivi;
  int head_dim;
  bool any_blocks;
};

kvk_status prepare(const kvk_table* t, int32_t l0, int32_t l1, const void* q, int32_t q_dtype,
                   int32_t n_stored, float scale, const void* w_uk, const void* w_uv, const void* arena,
                   float* out, void* workspace, size_t ws_bytes, DecodePlan& P) {
  if (!t) return fail(KVK_ERR_INVALID, "decode: NULL table");
  const kvk_dims& d = t->d;
  if (l0 < 0 || l1 > d.n_layers || l0 >= l1)
    return fail(KVK_ERR_INVALID, "layer range [%d, %d) invalid for %d layers", l0, l1, d.n_layers);
  if (!q || !arena || !out || !workspace) return fail(KVK_ERR_INVALID, "NULL buffer");
  if (w_uk || w_uv) return fail(KVK_ERR_INVALID, "w_uk / w_uv must be NULL for a GQA table");
  if (q_dtype != KVK_BF16 && q_dtype != KVK_F32) return fail(KVK_ERR_INVALID, "q_dtype %d", q_dtype);
  if (n_stored < 0 || n_stored > t->cap)
    return fail(KVK_ERR_INVALID, "n_stored %d outside 0..%d", n_stored, t->cap);
  if (!(scale == scale)) return fail(KVK_ERR_INVALID, "scale is NaN");
  if ((reinterpret_cast<uintptr_t>(q) & 15) || (reinterpret_cast<uintptr_t>(arena) & 15) ||
      (reinterpret_cast<uintptr_t>(out) & 15) || (reinterpret_cast<uintptr_t>(workspace) & 255))
    return fail(KVK_ERR_INVALID, "misaligned buffer (q/arena/out 16 B, workspace 256 B)");

  const int32_t G = d.n_q_heads / d.n_kv_heads;
  const int32_t D = d.head_dim;
  const int32_t nbf = n_stored / KVK_GROUP, ntail = n_stored % KVK_GROUP;
  const int32_t nblk = nbf + (ntail > 0 ? 1 : 0);
  DecodeArgs& a = P.d1;
  CombineArgs& ca = P.c1;
  a.arena = static_cast<const uint8_t*>(arena);
  a.q = q;
  a.ws = static_cast<float*>(workspace);
  a.q_f32 = q_dtype == KVK_F32;
  a.B = d.batch;
  a.Hq = d.n_q_heads;
  a.Hkv = d.n_kv_heads;
  a.G = G;
  a.nbf = nbf;
  a.ntail = ntail;
  a.nb_cap = t->nb_cap;
  a.scale_log2 = scale * kLog2e;
  a.n_items = 0;
  ca.out = out;
  ca.ws = static_cast<const float*>(workspace);
  ca.B = d.batch;
  ca.Hq = d.n_q_heads;
  ca.Hkv = d.n_kv_heads;
  ca.G = G;
  ca.n_layers = l1 - l0;
  ca.n_rows = (l1 - l0) * d.batch * d.n_q_heads;

  // One work item per distinct anchor read by the range (§2.1 depth sharing).
  int item_of_anchor[KVK_MAX_LAYERS];
  for (int l = 0; l < KVK_MAX_LAYERS; ++l) item_of_anchor[l] = -1;
  int64_t ws_floats = 0, waves = 0;
  for (int l = l0; l < l1; ++l) {
    const int anc = t->info.anchor_of[l];
    if (item_of_anchor[anc] < 0) {
      const int n = a.n_items++;
      DecodeItem& it = a.items[n];
      const int rb = anc > l0 ? anc : l0;
      const int re = t->next_anchor[anc] < l1 ? t->next_anchor[anc] : l1;
      it.region = t->info.layer_offset[anc];
      it.stream_bytes = (int32_t)t->info.stream_bytes[anc];
      it.block_bytes = (int32_t)t->block_bytes[anc];
      it.bits = t->bits[anc];
      it.q_layer0 = rb - l0;
      it.geff = G * (re - rb);
      it.split_blocks = split_blocks_for(it.bits, d.qscheme, D);
      it.nsplit = n_splits(nblk, it.split_blocks);
      const int nch = (it.geff + 15) / 16;
      it.nchp = nch == 1 ? 1 : (nch == 2 ? 2 : 4);
      waves = (waves + 3) / 4 * 4;  // a chunk group never straddles a workgroup
      it.wave_begin = (int32_t)waves;
      waves += (int64_t)d.batch * d.n_kv_heads * it.nsplit * it.nchp;
      it.ws_off = (int32_t)ws_floats;
      ws_floats += (int64_t)d.batch * d.n_kv_heads * it.nsplit * it.geff * (D + 4);
      ca.item_ws_off[n] = it.ws_off;
      ca.item_nsplit[n] = it.nsplit;
      ca.item_geff[n] = it.geff;
      item_of_anchor[anc] = n;
    }
    const int ii = item_of_anchor[anc];
    ca.layer_item[l - l0] = ii;
    ca.layer_slot0[l - l0] = (l - l0 - a.items[ii].q_layer0) * G;
  }
  if ((size_t)ws_floats * sizeof(float) > ws_bytes)
    return fail(KVK_ERR_BUFFER, "workspace %zu bytes < %lld needed", ws_bytes,
                (long long)(ws_floats * sizeof(float)));
  if (ws_floats > 0x7fffffffLL) return fail(KVK_ERR_UNSUPPORTED, "workspace exceeds 2^31 floats");
  if (waves > 0x7ffffff0LL) return fail(KVK_ERR_UNSUPPORTED, "too many decode waves");
  a.total_waves = (int32_t)waves;
  P.kivi = d.qscheme == KVK_Q_KIVI32;
  P.head_dim = D;
  P.any_blocks = nblk > 0 && waves > 0;
  return KVK_OK;
}

kvk_status launch_d1(const DecodePlan& P, hipStream_t st) {
  if (!P.any_blocks) return KVK_OK;
  const unsigned grid = (unsigned)((P.d1.total_waves + 3) / 4);
  if (P.head_dim == 128) {
    if (P.kivi) hipLaunchKernelGGL((gqa_decode_kernel<128, true>), dim3(grid), dim3(256), 0, st, P.d1);
    else hipLaunchKernelGGL((gqa_decode_kernel<128, false>), dim3(grid), dim3(256), 0, st, P.d1);
  } else {
    if (P.kivi) hipLaunchKernelGGL((gqa_decode_kernel<64, true>), dim3(grid), dim3(256), 0, st, P.d1);
    else hipLaunchKernelGGL((gqa_decode_kernel<64, false>), dim3(grid), dim3(256), 0, st, P.d1);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(KVK_ERR_DEVICE, "decode launch: %s", hipGetErrorString(e));
  return KVK_OK;
}

kvk_status launch_c1(const DecodePlan& P, hipStream_t st) {
  const unsigned grid = (unsigned)((P.c1.n_rows + 3) / 4);
  if (P.head_dim == 128) hipLaunchKernelGGL(gqa_combine_kernel<128>, dim3(grid), dim3(256), 0, st, P.c1);
  else hipLaunchKernelGGL(gqa_combine_kernel<64>, dim3(grid), dim3(256), 0, st, P.c1);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(KVK_ERR_DEVICE, "combine launch: %s", hipGetErrorString(e));
  return KVK_OK;
}

}  // namespace

extern "C" kvk_status kvk_decode_attention(const kvk_table* t, int32_t l0, int32_t l1, const void* q,
                                           int32_t q_dtype, int32_t n_stored, float scale,
                                           const void* w_uk, const void* w_uv, const void* arena,
                                           float* out, void* workspace, size_t ws_bytes,
                                           hipStream_t stream) {
  DecodePlan P;
  kvk_status st = prepare(t, l0, l1, q, q_dtype, n_stored, scale, w_uk, w_uv, arena, out, workspace,
                          ws_bytes, P);
  if (st != KVK_OK) return st;
  st = launch_d1(P, stream);
  if (st != KVK_OK) return st;
  return launch_c1(P, stream);
}

extern "C" kvk_status kvk_decode_splits(const kvk_table* t, int32_t l0, int32_t l1, const void* q,
                                        int32_t q_dtype, int32_t n_stored, float scale,
                                        const void* w_uk, const void* w_uv, const void* arena,
                                        void* workspace, size_t ws_bytes, hipStream_t stream) {
  DecodePlan P;
  float* dummy_out = static_cast<float*>(workspace);  // not written by this phase
  kvk_status st = prepare(t, l0, l1, q, q_dtype, n_stored, scale, w_uk, w_uv, arena, dummy_out,
                          workspace, ws_bytes, P);
  if (st != KVK_OK) return st;
  return launch_d1(P, stream);
}

extern "C" kvk_status kvk_decode_merge(const kvk_table* t, int32_t l0, int32_t l1, int32_t n_stored,
                                       const void* workspace, size_t ws_bytes, float* out,
                                       hipStream_t stream) {
  DecodePlan P;
  // q and arena are not read by the merge; the workspace stands in for them in validation.
  kvk_status st = prepare(t, l0, l1, workspace, KVK_F32, n_stored, 1.0f, nullptr, nullptr, workspace,
                          out, const_cast<void*>(workspace), ws_bytes, P);
  if (st != KVK_OK) return st;
  return launch_c1(P, stream);
}

extern "C" kvk_status kvk_read_bytes(const kvk_table* t, int32_t l0, int32_t l1, int32_t n_stored,
                                     int64_t* out_bytes) {
  if (!t || !out_bytes) return fail(KVK_ERR_INVALID, "kvk_read_bytes: NULL argument");
  const kvk_dims& d = t->d;
  if (l0 < 0 || l1 > d.n_layers || l0 >= l1)
    return fail(KVK_ERR_INVALID, "layer range [%d, %d) invalid for %d layers", l0, l1, d.n_layers);
  if (n_stored < 0 || n_stored > t->cap)
    return fail(KVK_ERR_INVALID, "n_stored %d outside 0..%d", n_stored, t->cap);
  bool seen[KVK_MAX_LAYERS] = {false};
  int64_t total = 0;
  const int64_t per_stream_tail = (int64_t)(n_stored % KVK_GROUP) * 4 * d.head_dim;
  for (int l = l0; l < l1; ++l) {
    const int a = t->info.anchor_of[l];
    if (seen[a]) continue;
    seen[a] = true;
    const int64_t per = (int64_t)(n_stored / KVK_GROUP) * t->block_bytes[a] + per_stream_tail;
    total += per * d.batch * d.n_kv_heads;
  }
  *out_bytes = total;
  return KVK_OK;
}
