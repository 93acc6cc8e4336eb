// Decode-step attention over per-layer compressed GQA caches (D1 + C1).
//
// KV-Kaizen §2.1: every layer attends with its own query over the keys and values
// of its anchor (itself, or the nearest earlier producing layer).  Layers that
// share an anchor are served together: their query rows are stacked so that the
// anchor's bytes are read once per step.  Decode is bound by reading the cache
// (§1), so the kernel streams each (sequence, KV head) stream once, split along
// the context into pieces of 1-16 MiB (the split rule is in table.cpp); a second
// kernel merges the splits by log-sum-exp.
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

#include <algorithm>
#include <mutex>
#include <vector>

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
  int32_t b0;            // first sequence of the item's streams
  int32_t nb;            // sequences of the item (all B, or one under per-sequence plans)
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
  const DecodeItem* items_dev;  // per-sequence plans: the work list in device memory
  const uint64_t* list_hdr;     // per-sequence plans: its header (magic, hash)
  uint64_t list_hash;           // the hash this call's list must carry
  DecodeItem items[kMaxItems];  // one plan: the work list in the arguments
};
static_assert(sizeof(DecodeArgs) <= 4096, "kernel arguments");

// Combine-side fields of a work item (device memory, per-sequence plans).
struct CombItem {
  int64_t tail;  // byte offset of stream 0's tail block of the item
  int32_t ws_off, nsplit, geff, stream_bytes, b0, split_blocks;
};

// Header of a per-sequence work list in the workspace: a magic word and the hash
// of the list that follows.  A kernel whose arguments expect another hash (a
// workspace never set up, or set up for another table or layer range) touches
// nothing through the list.
constexpr uint64_t kListMagic = 0x4b564b4c49535431ull;  // "KVKLIST1"

struct CombineArgs {
  float* out;
  const float* ws;
  const uint8_t* arena;
  const void* q;
  int32_t q_f32;
  float scale_log2;
  int32_t ntail;   // tokens in the bf16 tail block
  int32_t nb_cap;
  int32_t B, Hq, Hkv, G;
  int32_t n_rows;  // layers * B * Hq
  int32_t n_layers;
  int64_t item_tail[kMaxItems];  // byte offset of stream 0's tail block of each item
  int32_t item_stream_bytes[kMaxItems];
  int32_t layer_item[kMaxItems];
  int32_t layer_slot0[kMaxItems];
  int32_t item_ws_off[kMaxItems];
  int32_t item_nsplit[kMaxItems];
  int32_t item_geff[kMaxItems];
  const CombItem* citems;  // per-sequence plans: per item, and per (layer, sequence)
  const int32_t* map;      // the item and the first query slot of the row group
  const uint64_t* list_hdr;
  uint64_t list_hash;
  int32_t nbf;             // full blocks stored per stream (per-sequence plans: live splits)
};

__device__ __forceinline__ f4 mfma16(half8 a, half8 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f4 mfmab(bf16x8 a, bf16x8 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float wave_max_kg(float x) { return rows_max(x); }
__device__ __forceinline__ float wave_sum_kg(float x) { return rows_sum(x); }

__device__ __forceinline__ bf16x8 to_bf16x8(const float* x) {
  bf16x8 r;
#pragma unroll
  for (int s = 0; s < 8; ++s) r[s] = (__bf16)x[s];
  return r;
}

// ---------------------------------------------------------------------------
// Per-lane raw bytes of one 32-token block, loaded ahead of use.
// ---------------------------------------------------------------------------

template <int D, int BITS, int QS>
struct Raw {
  static constexpr int KB = BITS == 16 ? D / 2 : D * BITS / 32;  // bytes per lane per K tile
  static constexpr int VB = BITS == 16 ? D : D * BITS / 16;      // bytes per lane of V
  static constexpr int MB = BITS == 16 ? 0 : (QS == kQsKivi ? D / 8 : (QS == kQsG64 ? D / 16 : 32));  // metadata bytes per lane
  uint32_t k[2][KB / 4];
  uint32_t v[VB / 4];
  uint32_t m[MB > 0 ? MB / 4 : 1];
};

// Stream loads go through a buffer resource whose range ends at the last byte of
// the split: a prefetch past the split returns zeros without touching memory (the
// range check covers the vector and the scalar offset together; checked on
// gfx950 with an in-bounds probe), so the prefetch ring is reloaded without
// branches and the compiler can count the outstanding loads exactly (a branch
// around a reload makes it wait for all of them).
typedef __amdgpu_buffer_rsrc_t Rsrc;

__device__ __forceinline__ Rsrc stream_rsrc(const uint8_t* base, int nbytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(base), (short)0, nbytes, 0x00020000);
}

// voff: the lane's byte offset inside the part (a vector register shared by all
// blocks); soff: the block and part offset (a scalar register).
template <int N, int POL>
__device__ __forceinline__ void load_words(Rsrc rs, int voff, int soff, uint32_t* w) {
  if constexpr (N % 4 == 0) {
#pragma unroll
    for (int i = 0; i < N / 4; ++i) {
      const u4v x = __builtin_amdgcn_raw_buffer_load_b128(rs, voff + 16 * i, soff, POL);
      w[4 * i] = x[0]; w[4 * i + 1] = x[1]; w[4 * i + 2] = x[2]; w[4 * i + 3] = x[3];
    }
  } else if constexpr (N == 2) {
    const u2v x = __builtin_amdgcn_raw_buffer_load_b64(rs, voff, soff, POL);
    w[0] = x[0]; w[1] = x[1];
  } else {
    w[0] = __builtin_amdgcn_raw_buffer_load_b32(rs, voff, soff, POL);
  }
}

// The lane's share of a part (N words at soff, share_byte rules): shares above 16
// bytes are dealt out in 16-byte pieces, so each load of the wave reads 1 KiB.
template <int N, int POL>
__device__ __forceinline__ void load_share(Rsrc rs, int lane, int soff, uint32_t* w) {
  if constexpr (N % 4 == 0) {
#pragma unroll
    for (int i = 0; i < N / 4; ++i) {
      const u4v x = __builtin_amdgcn_raw_buffer_load_b128(rs, 16 * lane, soff + 1024 * i, POL);
      w[4 * i] = x[0]; w[4 * i + 1] = x[1]; w[4 * i + 2] = x[2]; w[4 * i + 3] = x[3];
    }
  } else {
    load_words<N, POL>(rs, 4 * N * lane, soff, w);
  }
}

// Loads of the block at byte offset `blk` (wave-uniform) of the stream (block
// layout of include/kvk.h), in the parts that are consumed at different times:
// key codes (score phase), value codes (value phase), metadata.
template <int D, int BITS, int QS, int POL>
__device__ __forceinline__ void load_k(Raw<D, BITS, QS>& r, Rsrc rs, int blk, int lane) {
  using R = Raw<D, BITS, QS>;
  constexpr int tile = BITS == 16 ? 32 * D : 2 * D * BITS;
#pragma unroll
  for (int tau = 0; tau < 2; ++tau) load_share<R::KB / 4, POL>(rs, lane, blk + tau * tile, r.k[tau]);
}

template <int D, int BITS, int QS, int POL>
__device__ __forceinline__ void load_v(Raw<D, BITS, QS>& r, Rsrc rs, int blk, int lane) {
  using R = Raw<D, BITS, QS>;
  constexpr int vbase = BITS == 16 ? 64 * D : 4 * D * BITS;
  load_share<R::VB / 4, POL>(rs, lane, blk + vbase, r.v);
}

// KIVI32 / GROUP64: the lane's share of the 8D- / 4D-byte metadata area.  SYMROW:
// part 0 the K row scales (m[0..3]), part 1 the V row scales (m[4..7]) of the
// lane's tokens.
template <int D, int BITS, int QS, int POL>
__device__ __forceinline__ void load_m(Raw<D, BITS, QS>& r, Rsrc rs, int blk, int lane, int part) {
  using R = Raw<D, BITS, QS>;
  if constexpr (BITS != 16) {
    const int meta = blk + 8 * D * BITS;
    if constexpr (QS != kQsSym) {
      load_share<R::MB / 4, POL>(rs, lane, meta, r.m);
    } else {
      const int kg = lane >> 4;
#pragma unroll
      for (int tau = 0; tau < 2; ++tau)
        load_words<2, POL>(rs, 8 * kg, meta + 64 * part + 32 * tau, r.m + 4 * part + 2 * tau);
    }
  }
}

template <int D, int BITS, int QS, int POL>
__device__ __forceinline__ void load_raw(Raw<D, BITS, QS>& r, Rsrc rs, int blk, int lane) {
  load_k<D, BITS, QS, POL>(r, rs, blk, lane);
  load_v<D, BITS, QS, POL>(r, rs, blk, lane);
  load_m<D, BITS, QS, POL>(r, rs, blk, lane, 0);
  if constexpr (QS == kQsSym) load_m<D, BITS, QS, POL>(r, rs, blk, lane, 1);
}

// Unpack the 8 codes (one MFMA k-step) of chunk x from a lane's code words.
template <int BITS>
__device__ __forceinline__ half8 unpack_chunk(const uint32_t* w, int x, float off) {
  if constexpr (BITS == 4) {
    return unpack4(w[x], off);
  } else if constexpr (BITS == 8) {
    return unpack8(w[2 * x], w[2 * x + 1], off);
  } else {
    return unpack2_half(w[x >> 1] >> (8 * (x & 1)), off);
  }
}

// ---------------------------------------------------------------------------
// Per-wave state of one work unit (16 query rows: lane row = lane % 16).
// ---------------------------------------------------------------------------

template <int D>
struct State {
  static constexpr int NJ = D / 32;  // MFMA k-steps over channels
  static constexpr int NM = D / 16;  // value channel tiles
  static constexpr int NG = D / 32;  // value channel groups (KIVI32)
  f4 o[NM];                          // O^T tiles
  float m;                           // running max, log2 domain
  float l;                           // lane-partial running sum
};

// Extra accumulators rescaled with the output: the value zero-point sums of the
// grouped schemes (one per channel group).
template <int N>
struct Extra {
  f4 zo[N];
};

template <int D, int NX>
__device__ __forceinline__ void softmax_update(State<D>& u, Extra<NX>& ex, float (&x)[8]) {
  float mb = x[0];
#pragma unroll
  for (int e = 1; e < 8; ++e) mb = fmaxf(mb, x[e]);
  mb = wave_max_kg(mb);
  // The first block of a unit is always a stored block, so mnew is finite from
  // then on: the first alpha is 2^-inf = 0 and masked logits give p = 0.
  const float mnew = fmaxf(u.m, mb);
  const float alpha = __builtin_amdgcn_exp2f(u.m - mnew);
  float ps = 0.0f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float p = __builtin_amdgcn_exp2f(x[e] - mnew);
    x[e] = p;
    ps += p;
  }
  u.l = u.l * alpha + ps;
  u.m = mnew;
  if (__any(alpha != 1.0f)) {
#pragma unroll
    for (int mt = 0; mt < State<D>::NM; ++mt) u.o[mt] *= alpha;
#pragma unroll
    for (int g = 0; g < NX; ++g) ex.zo[g] *= alpha;
  }
}

__device__ __forceinline__ half8 to_half8(const float (&x)[8]) {
  half8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = (_Float16)x[e];
  return r;
}

// A bf16 block (b = 16 layers).
// Each compute_* function consumes ring entry `r` and, with RELOAD, refills each
// part of it from the block at byte offset `next` as soon as that part has been
// read, so that the registers stay in flight for as long as possible.
template <int D, int QS, bool RELOAD, int POL>
__device__ __forceinline__ void compute_bf16(State<D>& u, const bf16x8 (&qbh)[D / 32],
                                             const bf16x8 (&qbl)[D / 32], Raw<D, 16, QS>& r, Rsrc rs,
                                             int next, bool valid, int lane) {
  constexpr int NJ = D / 32, NM = D / 16;
  const int kg = lane >> 4;
  float x[8];
#pragma unroll
  for (int tau = 0; tau < 2; ++tau) {
    f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const u4v w = {r.k[tau][4 * j], r.k[tau][4 * j + 1], r.k[tau][4 * j + 2], r.k[tau][4 * j + 3]};
      const bf16x8 kop = bitcast<bf16x8>(w);
      acc = mfmab(kop, qbh[j], acc);
      acc = mfmab(kop, qbl[j], acc);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) x[4 * tau + e] = valid ? acc[e] : -INFINITY;  // q carries scale*log2(e)
  }
  if constexpr (RELOAD) {
    __builtin_amdgcn_sched_barrier(0);  // the refill may not rise above the reads it replaces
    load_k<D, 16, QS, POL>(r, rs, next, lane);
  }
  Extra<0> none;
  softmax_update<D, 0>(u, none, x);
  float h[8], lw[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    h[e] = (float)(__bf16)x[e];
    lw[e] = x[e] - h[e];
  }
  const bf16x8 phi = to_bf16x8(h), plo = to_bf16x8(lw);
#pragma unroll
  for (int mt = 0; mt < NM; ++mt) {
    const u4v w = {r.v[4 * mt], r.v[4 * mt + 1], r.v[4 * mt + 2], r.v[4 * mt + 3]};
    const bf16x8 vop = bitcast<bf16x8>(w);
    u.o[mt] = mfmab(vop, phi, u.o[mt]);
    u.o[mt] = mfmab(vop, plo, u.o[mt]);
  }
  if constexpr (RELOAD) {
    __builtin_amdgcn_sched_barrier(0);
    load_v<D, 16, QS, POL>(r, rs, next, lane);
  }
}

// KIVI32 block of BITS-bit codes.  The block's metadata goes through the wave's
// LDS slot so that the 16 lanes sharing a channel (or token) group read it by
// broadcast.
template <int D, int BITS, bool RELOAD, int POL>
__device__ __forceinline__ void compute_kivi(State<D>& u, Extra<D / 32>& ex, const half8 (&qh)[D / 32],
                                             const half8 (&ql)[D / 32], Raw<D, BITS, kQsKivi>& r, Rsrc rs,
                                             int next, bool valid, uint32_t* lds, int lane) {
  using R = Raw<D, BITS, kQsKivi>;
  constexpr int NJ = D / 32, NG = D / 32;
  const int kg = lane >> 4;
#pragma unroll
  for (int i = 0; i < R::MB / 4; ++i) lds[lane * (R::MB / 4) + i] = r.m[i];
  if constexpr (RELOAD) {
    __builtin_amdgcn_sched_barrier(0);
    load_m<D, BITS, kQsKivi, POL>(r, rs, next, lane, 0);
  }
  const half8* kmeta = reinterpret_cast<const half8*>(lds);  // scale[D], zero[D], V meta[2D]
  // K: S = sum_c (q_c s_c) u_c + sum_c q_c z_c.  q' = q s as fp16 hi + lo (error-free
  // product of the fp16 hi part, rounded sum with the lo part).
  f4 zt = {0.f, 0.f, 0.f, 0.f};
  f4 acc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const half8 sv = kmeta[4 * j + kg];          // scales of channels 32j + 8kg + 0..7
    const half8 zv = kmeta[D / 8 + 4 * j + kg];  // zeros of the same channels
    const half8 hi = qh[j] * sv;
    const half8 err = __builtin_elementwise_fma(qh[j], sv, -hi);
    const half8 lo = __builtin_elementwise_fma(ql[j], sv, err);
    zt = mfma16(zv, qh[j], zt);  // every token row gets sum_c z_c q_c
    zt = mfma16(zv, ql[j], zt);
#pragma unroll
    for (int tau = 0; tau < 2; ++tau) {
      const half8 kop = unpack_chunk<BITS>(r.k[tau], j, 0.0f);
      acc[tau] = mfma16(kop, hi, acc[tau]);
      acc[tau] = mfma16(kop, lo, acc[tau]);
    }
    __builtin_amdgcn_sched_barrier(0);  // keep one k-step's operands live at a time
  }
  if constexpr (RELOAD) {
    __builtin_amdgcn_sched_barrier(0);
    load_k<D, BITS, kQsKivi, POL>(r, rs, next, lane);
  }
  float x[8];
#pragma unroll
  for (int tau = 0; tau < 2; ++tau)
#pragma unroll
    for (int e = 0; e < 4; ++e) x[4 * tau + e] = valid ? acc[tau][e] + zt[e] : -INFINITY;
  softmax_update<D, D / 32>(u, ex, x);
  const half8 p = to_half8(x);
  // V: o_c = sum_t (p_t s_tg) u_tc + sum_t p_t z_tg, g = c / 32.  At 2 and 4 bits
  // the value codes enter raw (1024 + u / c per slot, raw_codes), the probabilities
  // carry the slot factors c, and 1024 sum_t c_t p_t s_tg comes off in the same
  // block through one more product per channel tile, so the accumulators never hold
  // the 1024 offset across blocks (fp32 rounding stays relative to the block's own
  // mass).  At 8 bits the unpacking fix-up is cheap and the path is bound by HBM.
  const half8* vmeta = kmeta + D / 4;
  const half8 pc = BITS == 8 ? p : p * raw_factors<BITS>();
  const _Float16 m1024 = (_Float16)-1024.0f;
  const half8 neg = {m1024, m1024, m1024, m1024, m1024, m1024, m1024, m1024};
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const half8 vs = vmeta[(g * 2 + 0) * 4 + kg];
    const half8 vz = vmeta[(g * 2 + 1) * 4 + kg];
    const half8 ps = pc * vs;
    ex.zo[g] = mfma16(vz, p, ex.zo[g]);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int mt = 2 * g + h;
      if constexpr (BITS == 8) {
        u.o[mt] = mfma16(unpack_chunk<BITS>(r.v, mt, 0.0f), ps, u.o[mt]);
      } else {
        const uint32_t w0 = BITS == 4 ? r.v[mt] : r.v[mt >> 1] >> (8 * (mt & 1));
        u.o[mt] = mfma16(neg, ps, u.o[mt]);
        u.o[mt] = mfma16(raw_codes<BITS>(w0, 0u), ps, u.o[mt]);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  }
  if constexpr (RELOAD) {
    __builtin_amdgcn_sched_barrier(0);
    load_v<D, BITS, kQsKivi, POL>(r, rs, next, lane);
  }
}

// SYMROW block: per-token scales factor out of both contractions.
template <int D, int BITS, bool RELOAD, int POL>
__device__ __forceinline__ void compute_symrow(State<D>& u, const half8 (&qh)[D / 32],
                                               const half8 (&ql)[D / 32], Raw<D, BITS, kQsSym>& r,
                                               Rsrc rs, int next, bool valid, int lane) {
  constexpr int NJ = D / 32, NM = D / 16;
  const float off = (float)(1 << (BITS - 1));
  float x[8];
#pragma unroll
  for (int tau = 0; tau < 2; ++tau) {
    f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const half8 kop = unpack_chunk<BITS>(r.k[tau], j, off);
      acc = mfma16(kop, qh[j], acc);
      acc = mfma16(kop, ql[j], acc);
    }
    const uint32_t s01 = r.m[2 * tau], s23 = r.m[2 * tau + 1];
    const float sk[4] = {__uint_as_float(s01 << 16), __uint_as_float(s01 & 0xffff0000u),
                         __uint_as_float(s23 << 16), __uint_as_float(s23 & 0xffff0000u)};
#pragma unroll
    for (int e = 0; e < 4; ++e) x[4 * tau + e] = valid ? acc[e] * sk[e] : -INFINITY;
  }
  if constexpr (RELOAD) {
    __builtin_amdgcn_sched_barrier(0);
    load_k<D, BITS, kQsSym, POL>(r, rs, next, lane);
    load_m<D, BITS, kQsSym, POL>(r, rs, next, lane, 0);
  }
  Extra<0> none;
  softmax_update<D, 0>(u, none, x);
  float ps[8];
#pragma unroll
  for (int tau = 0; tau < 2; ++tau) {
    const uint32_t s01 = r.m[4 + 2 * tau], s23 = r.m[5 + 2 * tau];
    ps[4 * tau + 0] = x[4 * tau + 0] * __uint_as_float(s01 << 16);
    ps[4 * tau + 1] = x[4 * tau + 1] * __uint_as_float(s01 & 0xffff0000u);
    ps[4 * tau + 2] = x[4 * tau + 2] * __uint_as_float(s23 << 16);
    ps[4 * tau + 3] = x[4 * tau + 3] * __uint_as_float(s23 & 0xffff0000u);
  }
  const half8 p = to_half8(ps);
  if constexpr (RELOAD) {
    __builtin_amdgcn_sched_barrier(0);
    load_m<D, BITS, kQsSym, POL>(r, rs, next, lane, 1);
  }
#pragma unroll
  for (int mt = 0; mt < NM; ++mt) u.o[mt] = mfma16(unpack_chunk<BITS>(r.v, mt, off), p, u.o[mt]);
  if constexpr (RELOAD) {
    __builtin_amdgcn_sched_barrier(0);
    load_v<D, BITS, kQsSym, POL>(r, rs, next, lane);
  }
}

// GROUP64 block: per (token, 64-channel group) scale and zero for keys and values.
// The metadata goes through the wave's LDS slot as for KIVI32.  Keys: the codes
// enter the products raw, one accumulator per channel group, and
//   S_t = sum_g s_tg (sum_{c in g} q_c u_tc) + z_tg Q_g,   Q_g = sum_{c in g} q_c
// (Q_g per query row, computed once per unit).  Values: as KIVI32's, with groups of
// 64 channels (four channel tiles per group).
template <int D, int BITS, bool RELOAD, int POL>
__device__ __forceinline__ void compute_g64(State<D>& u, Extra<D / 64>& ex, const half8 (&qh)[D / 32],
                                            const half8 (&ql)[D / 32], const float (&qsum)[D / 64],
                                            Raw<D, BITS, kQsG64>& r, Rsrc rs, int next, bool valid, uint32_t* lds,
                                            int lane) {
  using R = Raw<D, BITS, kQsG64>;
  constexpr int NJ = D / 32, NG = D / 64;
  const int kg = lane >> 4;
#pragma unroll
  for (int i = 0; i < R::MB / 4; ++i) lds[lane * (R::MB / 4) + i] = r.m[i];
  if constexpr (RELOAD) {
    __builtin_amdgcn_sched_barrier(0);
    load_m<D, BITS, kQsG64, POL>(r, rs, next, lane, 0);
  }
  const _Float16* meta = reinterpret_cast<const _Float16*>(lds);  // K meta [D halves], V meta [D halves]
  f4 acc[2][NG];
#pragma unroll
  for (int tau = 0; tau < 2; ++tau)
#pragma unroll
    for (int g = 0; g < NG; ++g) acc[tau][g] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
#pragma unroll
    for (int tau = 0; tau < 2; ++tau) {
      const half8 kop = unpack_chunk<BITS>(r.k[tau], j, 0.0f);
      acc[tau][j / 2] = mfma16(kop, qh[j], acc[tau][j / 2]);
      acc[tau][j / 2] = mfma16(kop, ql[j], acc[tau][j / 2]);
    }
    __builtin_amdgcn_sched_barrier(0);  // keep one k-step's operands live at a time
  }
  if constexpr (RELOAD) {
    __builtin_amdgcn_sched_barrier(0);
    load_k<D, BITS, kQsG64, POL>(r, rs, next, lane);
  }
  float x[8];
#pragma unroll
  for (int tau = 0; tau < 2; ++tau) {
    float sc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      // scales then zeros of tokens 16 tau + 4 kg + e, e = 0..3
      const half8 sz = *reinterpret_cast<const half8*>(meta + ((tau * 4 + kg) * NG * 2 + g * 2) * 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) sc[e] += (float)sz[e] * acc[tau][g][e] + (float)sz[4 + e] * qsum[g];
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) x[4 * tau + e] = valid ? sc[e] : -INFINITY;
  }
  softmax_update<D, NG>(u, ex, x);
  const half8 p = to_half8(x);
  // V: o_c = sum_t (p_t s_tg) u_tc + sum_t p_t z_tg, g = c / 64 (raw codes at 2 and 4
  // bits as for KIVI32).
  const half8* vmeta = reinterpret_cast<const half8*>(meta + D);
  const half8 pc = BITS == 8 ? p : p * raw_factors<BITS>();
  const _Float16 m1024 = (_Float16)-1024.0f;
  const half8 neg = {m1024, m1024, m1024, m1024, m1024, m1024, m1024, m1024};
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const half8 vs = vmeta[(g * 2 + 0) * 4 + kg];
    const half8 vz = vmeta[(g * 2 + 1) * 4 + kg];
    const half8 ps = pc * vs;
    ex.zo[g] = mfma16(vz, p, ex.zo[g]);
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      const int mt = 4 * g + h;
      if constexpr (BITS == 8) {
        u.o[mt] = mfma16(unpack_chunk<BITS>(r.v, mt, 0.0f), ps, u.o[mt]);
      } else {
        const uint32_t w0 = BITS == 4 ? r.v[mt] : r.v[mt >> 1] >> (8 * (mt & 1));
        u.o[mt] = mfma16(neg, ps, u.o[mt]);
        u.o[mt] = mfma16(raw_codes<BITS>(w0, 0u), ps, u.o[mt]);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  }
  if constexpr (RELOAD) {
    __builtin_amdgcn_sched_barrier(0);
    load_v<D, BITS, kQsG64, POL>(r, rs, next, lane);
  }
}

// Blocks kept in flight per wave (registers); the host rounds split lengths to a
// multiple of this depth.
template <int BITS>
constexpr int ring_depth() {
  return kvk::gqa_ring_depth(BITS);
}

// The query as fp16 hi + lo (integer-code paths) and as bf16 hi + lo (bf16 blocks).
template <int D>
__device__ __forceinline__ void split_bf16(const half8 (&qh)[D / 32], const half8 (&ql)[D / 32],
                                           bf16x8 (&qbh)[D / 32], bf16x8 (&qbl)[D / 32]) {
#pragma unroll
  for (int j = 0; j < D / 32; ++j) {
    float hb[8], lb[8];
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const float q = (float)qh[j][s] + (float)ql[j][s];
      hb[s] = (float)(__bf16)q;
      lb[s] = q - hb[s];
    }
    qbh[j] = to_bf16x8(hb);
    qbl[j] = to_bf16x8(lb);
  }
}

// Load the lane's query row times scale * log2(e), as fp16 hi + lo (~22 significant
// bits), so that the score MFMAs produce base-2 logits directly.
template <int D>
__device__ __forceinline__ void load_query(const DecodeArgs& a, const DecodeItem& it, int row, int b, int kvh,
                                           int kg, half8 (&qh)[D / 32], half8 (&ql)[D / 32]) {
  const bool valid = row < it.geff;
  const int r = row / a.G, gh = row % a.G;
  const int64_t qrow = (((int64_t)(it.q_layer0 + r) * a.B + b) * a.Hq + kvh * a.G + gh) * D;
#pragma unroll
  for (int j = 0; j < D / 32; ++j) {
    const int ch = 32 * j + 8 * kg;
    float q[8];
    if (!valid) {
#pragma unroll
      for (int s = 0; s < 8; ++s) q[s] = 0.0f;
    } else if (a.q_f32) {
      const float4* qp = reinterpret_cast<const float4*>(static_cast<const float*>(a.q) + qrow + ch);
      const float4 v0 = qp[0], v1 = qp[1];
      q[0] = v0.x; q[1] = v0.y; q[2] = v0.z; q[3] = v0.w;
      q[4] = v1.x; q[5] = v1.y; q[6] = v1.z; q[7] = v1.w;
    } else {
      const uint4 v = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(a.q) + qrow + ch);
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        q[2 * p] = __uint_as_float(w[p] << 16);
        q[2 * p + 1] = __uint_as_float(w[p] & 0xffff0000u);
      }
    }
    float h16[8], l16[8];
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const float qs = q[s] * a.scale_log2;
      h16[s] = (float)(_Float16)qs;
      l16[s] = qs - h16[s];
    }
    qh[j] = to_half8(h16);
    ql[j] = to_half8(l16);
  }
}

// One work unit: 16 query rows over blocks [k0, k1) of one stream, ending with the
// split partial (o[D], m, l) of every valid row.  Everything the unit keeps in
// registers is local to this function, so that each precision gets its own
// register allocation.
template <int D, int BITS, int QS, int POL>
__device__ __forceinline__ void run_unit(const DecodeArgs& a, const DecodeItem& it, int sidx, int split,
                                         int chunk, uint32_t* lds, int lane) {
  constexpr int NR = ring_depth<BITS>();
  constexpr int NM = D / 16;
  constexpr int NX = BITS == 16 ? 0 : (QS == kQsKivi ? D / 32 : (QS == kQsG64 ? D / 64 : 0));
  const int b = it.b0 + sidx / a.Hkv, kvh = sidx % a.Hkv;  // sidx: the item's own stream index
  const int i16 = lane & 15, kg = lane >> 4;
  const int row = 16 * chunk + i16;
  const int k0 = split * it.split_blocks;
  const int k1 = min(a.nbf, k0 + it.split_blocks);
  const uint8_t* stream = a.arena + it.region + (int64_t)sidx * it.stream_bytes;
  State<D> u;
  u.m = -INFINITY;
  u.l = 0.0f;
#pragma unroll
  for (int mt = 0; mt < NM; ++mt) u.o[mt] = f4{0.f, 0.f, 0.f, 0.f};
  Extra<NX> ex;
#pragma unroll
  for (int g = 0; g < NX; ++g) ex.zo[g] = f4{0.f, 0.f, 0.f, 0.f};
  const int bb = it.block_bytes;
  const Rsrc rs = stream_rsrc(stream, k1 * bb);  // loads past block k1-1 read zeros
  Raw<D, BITS, QS> ring[NR];
#pragma unroll
  for (int i = 0; i < NR; ++i) load_raw<D, BITS, QS, POL>(ring[i], rs, (k0 + i) * bb, lane);
  // The query is issued after the ring so that both are waited for together.
  half8 qh[D / 32], ql[D / 32];
  load_query<D>(a, it, row, b, kvh, kg, qh, ql);
  bf16x8 qbh[D / 32], qbl[D / 32];
  if constexpr (BITS == 16) split_bf16<D>(qh, ql, qbh, qbl);
  float qsum[D / 64] = {};  // GROUP64: the row's query sum over each 64-channel group
  if constexpr (QS == kQsG64 && BITS != 16) {
#pragma unroll
    for (int j = 0; j < D / 32; ++j)
#pragma unroll
      for (int e = 0; e < 8; ++e) qsum[j / 2] += (float)qh[j][e] + (float)ql[j][e];
#pragma unroll
    for (int g = 0; g < D / 64; ++g) qsum[g] = wave_sum_kg(qsum[g]);
  }

  // Every reload is unconditional: ring entries past block k1-1 read zeros, and the
  // blocks they stand for (only in a stream's last split, since splits are a
  // multiple of NR blocks) enter with masked logits.
  for (int k = k0; k < k1; k += NR) {
#pragma unroll
    for (int i = 0; i < NR; ++i) {
      const int next = (k + i + NR) * bb;
      const bool valid = k + i < k1;
      if constexpr (BITS == 16) compute_bf16<D, QS, true, POL>(u, qbh, qbl, ring[i], rs, next, valid, lane);
      else if constexpr (QS == kQsKivi) compute_kivi<D, BITS, true, POL>(u, ex, qh, ql, ring[i], rs, next, valid, lds, lane);
      else if constexpr (QS == kQsG64)
        compute_g64<D, BITS, true, POL>(u, ex, qh, ql, qsum, ring[i], rs, next, valid, lds, lane);
      else compute_symrow<D, BITS, true, POL>(u, qh, ql, ring[i], rs, next, valid, lane);
    }
  }

  // partial: (o[D], m, l, pad, pad) per row
  float* base = a.ws + it.ws_off + ((int64_t)sidx * it.nsplit + split) * it.geff * (D + 4);
  const float lt = wave_sum_kg(u.l);
  if (row < it.geff) {
    float* pr = base + (int64_t)row * (D + 4);
#pragma unroll
    for (int mt = 0; mt < NM; ++mt) {
      f4 o = u.o[mt];
      if constexpr (NX > 0) o += ex.zo[mt / (NM / NX)];  // value zero-point sums of the channel group
      *reinterpret_cast<f4*>(pr + 16 * mt + 4 * kg) = o;
    }
    if (kg == 0) {
      pr[D] = u.m;
      pr[D + 1] = lt;
    }
  }
}

template <bool BATCHED>
__device__ __forceinline__ const DecodeItem& item_at(const DecodeArgs& a, int i) {
  if constexpr (BATCHED) return a.items_dev[i];
  else return a.items[i];
}

template <int D, int QS, bool BATCHED>
__global__ __launch_bounds__(256, 2) void gqa_decode_kernel(DecodeArgs a) {
  __shared__ uint32_t lds_meta[4][2 * D];  // per-wave metadata slot (KIVI32 8D bytes, GROUP64 4D)
  const int lane = threadIdx.x & 63;
  // Wave-uniform by construction; readfirstlane lets the compiler keep everything
  // derived from it (work item, stream address, buffer resource) in scalar registers.
  const int wslot = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wave = blockIdx.x * 4 + wslot;
  if (wave >= a.total_waves) return;
  if constexpr (BATCHED)
    if (a.list_hdr[0] != kListMagic || a.list_hdr[1] != a.list_hash) return;  // not this call's list
  int lo = 0, hi = a.n_items - 1;  // last item with wave_begin <= wave
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (item_at<BATCHED>(a, mid).wave_begin <= wave) lo = mid;
    else hi = mid - 1;
  }
  const DecodeItem& it = item_at<BATCHED>(a, lo);
  const int local = wave - it.wave_begin;
  int chunk, unit;
  if (it.nchp <= 4) {  // a unit's chunk waves share one workgroup
    chunk = local % it.nchp;
    unit = local / it.nchp;
  } else {
    // nchp = 4 k: a unit's waves fill k workgroups, which sit 8 apart in launch
    // order so that they land on one XCD and share the stream through its L2:
    // local workgroup j of a group of 8 units holds part j / 8 of unit j % 8.
    const int k = it.nchp >> 2, wl = local >> 2, j = wl % (8 * k);
    unit = wl / (8 * k) * 8 + j % 8;
    chunk = (j / 8) * 4 + (local & 3);
  }
  if (unit >= it.nb * a.Hkv * it.nsplit || 16 * chunk >= it.geff) return;  // alignment padding
  const int split = unit % it.nsplit;
  const int sidx = unit / it.nsplit;  // (b - b0) * Hkv + kvh
  // Per-sequence lists are laid out for the capacity: a split past the stored
  // blocks holds nothing at this n_stored (the merge reads only the live ones).
  if (BATCHED && split * it.split_blocks >= a.nbf) return;
  uint32_t* lds = lds_meta[wslot];
  // A stream read by one wave is streamed non-temporally; the waves of a stream read
  // by several row chunks read it through the caches (the later reads hit).
  if (it.nchp == 1) {
    switch (it.bits) {
      case 16: run_unit<D, 16, QS, kStreamPolicy>(a, it, sidx, split, chunk, lds, lane); break;
      case 8: run_unit<D, 8, QS, kStreamPolicy>(a, it, sidx, split, chunk, lds, lane); break;
      case 4: run_unit<D, 4, QS, kStreamPolicy>(a, it, sidx, split, chunk, lds, lane); break;
      default: run_unit<D, 2, QS, kStreamPolicy>(a, it, sidx, split, chunk, lds, lane); break;
    }
  } else {
    switch (it.bits) {
      case 16: run_unit<D, 16, QS, 0>(a, it, sidx, split, chunk, lds, lane); break;
      case 8: run_unit<D, 8, QS, 0>(a, it, sidx, split, chunk, lds, lane); break;
      case 4: run_unit<D, 4, QS, 0>(a, it, sidx, split, chunk, lds, lane); break;
      default: run_unit<D, 2, QS, 0>(a, it, sidx, split, chunk, lds, lane); break;
    }
  }
}

// Merge the splits of every output row by log-sum-exp, together with the bf16 tail
// tokens (fewer than 32), which this kernel attends to directly: one wave per
// (layer, b, head).
template <int D, bool BATCHED>
__global__ __launch_bounds__(256) void gqa_combine_kernel(CombineArgs a) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= a.n_rows) return;
  const int li = row / (a.B * a.Hq);
  const int rem = row % (a.B * a.Hq);
  const int b = rem / a.Hq, h = rem % a.Hq;
  int item, slot, nsplit, geff, ws_off, b0, sbytes;
  int64_t tail_off;
  int nlive;  // splits holding stored blocks (their partials are written)
  if constexpr (BATCHED) {
    if (a.list_hdr[0] != kListMagic || a.list_hdr[1] != a.list_hash) {  // not this call's list
      for (int e = lane; e < D; e += 64) a.out[(int64_t)row * D + e] = __builtin_nanf("");
      return;
    }
    const int32_t* m = a.map + ((int64_t)li * a.B + b) * 2;
    item = m[0];
    slot = m[1] + h % a.G;
    const CombItem& ci = a.citems[item];
    nsplit = ci.nsplit, geff = ci.geff, ws_off = ci.ws_off, b0 = ci.b0, sbytes = ci.stream_bytes;
    tail_off = ci.tail;
    nlive = min(nsplit, (a.nbf + ci.split_blocks - 1) / ci.split_blocks);
  } else {
    item = a.layer_item[li];
    slot = a.layer_slot0[li] + h % a.G;
    nsplit = a.item_nsplit[item], geff = a.item_geff[item], ws_off = a.item_ws_off[item], b0 = 0;
    sbytes = a.item_stream_bytes[item];
    tail_off = a.item_tail[item];
    nlive = nsplit;
  }
  const int kvh = h / a.G;
  const int sidx = (b - b0) * a.Hkv + kvh;  // the item's own stream index
  const float* base = a.ws + ws_off + (((int64_t)sidx * nsplit) * geff + slot) * (D + 4);
  const int64_t stride = (int64_t)geff * (D + 4);

  // tail scores: lane t < ntail takes token t
  const uint8_t* tail = a.arena + tail_off + (int64_t)sidx * sbytes;
  float st = -INFINITY;
  if (lane < a.ntail) {
    const int64_t qoff = (int64_t)row * D;
    float acc = 0.0f;
    for (int c0 = 0; c0 < D; c0 += 8) {
      const uint4 kw = *reinterpret_cast<const uint4*>(tail + k_bf16_byte(D, lane, c0));
      const uint32_t w[4] = {kw.x, kw.y, kw.z, kw.w};
      float q[8];
      if (a.q_f32) {
#pragma unroll
        for (int s = 0; s < 8; ++s) q[s] = static_cast<const float*>(a.q)[qoff + c0 + s];
      } else {
#pragma unroll
        for (int s = 0; s < 8; ++s) q[s] = bf16_to_f32(static_cast<const uint16_t*>(a.q)[qoff + c0 + s]);
      }
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        acc = fmaf(q[2 * p], __uint_as_float(w[p] << 16), acc);
        acc = fmaf(q[2 * p + 1], __uint_as_float(w[p] & 0xffff0000u), acc);
      }
    }
    st = acc * a.scale_log2;
  }
  float mstar = st;
  for (int s = lane; s < nlive; s += 64) mstar = fmaxf(mstar, base[s * stride + D]);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) mstar = fmaxf(mstar, __shfl_xor(mstar, off));
  constexpr int PER = D / 64;
  float acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) acc[e] = 0.0f;
  float lsum = 0.0f;
  for (int s = 0; s < nlive; ++s) {
    const float* p = base + s * stride;
    const float ms = p[D];
    const float w = (ms == -INFINITY) ? 0.0f : exp2f(ms - mstar);
    lsum = fmaf(w, p[D + 1], lsum);
#pragma unroll
    for (int e = 0; e < PER; ++e) acc[e] = fmaf(w, p[lane + 64 * e], acc[e]);
  }
  const float pt = (st == -INFINITY) ? 0.0f : exp2f(st - mstar);
  for (int t = 0; t < a.ntail; ++t) {
    const float w = __shfl(pt, t);
    lsum += w;
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const uint16_t vb = *reinterpret_cast<const uint16_t*>(tail + v_bf16_byte(D, t, lane + 64 * e));
      acc[e] = fmaf(w, bf16_to_f32(vb), acc[e]);
    }
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
// range in one launch) and the C1 arguments.  Under per-sequence plans the work
// list (one item per sequence and anchor: more than the arguments hold) lives at
// the head of the workspace, written there once by kvk_decode_setup; it is laid out
// for the capacity, so it does not depend on n_stored, and each call only checks
// that the setup of this table, layer range and workspace happened.
struct DecodePlan {
  DecodeArgs d1;
  CombineArgs c1;
  int qs;
  int head_dim;
  bool any_blocks;
  bool batched;
  std::vector<uint8_t> list;  // the host image of the work list (per-sequence plans)
  uint64_t hash;              // its hash (FNV-1a over the list after the header)
};

enum PrepareMode { kForDecode, kForSetup };

int64_t batched_items(const kvk_table* t, int32_t l0, int32_t l1) {
  int64_t n = 0;
  for (const kvk_table* s : t->seq) {
    bool seen[KVK_MAX_LAYERS] = {};
    for (int l = l0; l < l1; ++l) {
      const int a = s->info.anchor_of[l];
      if (!seen[a]) ++n;
      seen[a] = true;
    }
  }
  return n;
}

struct ListLayout {
  int64_t hdr, items, citems, map, total;  // byte offsets of the sections, and the size
};

ListLayout list_layout(const kvk_table* t, int32_t l0, int32_t l1) {
  const int64_t n = batched_items(t, l0, l1);
  ListLayout L;
  L.hdr = 0;
  L.items = 256;
  L.citems = L.items + round256(n * (int64_t)sizeof(DecodeItem));
  L.map = L.citems + round256(n * (int64_t)sizeof(CombItem));
  L.total = L.map + round256((int64_t)(l1 - l0) * t->d.batch * 2 * (int64_t)sizeof(int32_t));
  return L;
}

uint64_t fnv1a(const uint8_t* p, size_t n) {
  uint64_t h = 0xcbf29ce484222325ull;
  for (size_t i = 0; i < n; ++i) h = (h ^ p[i]) * 0x100000001b3ull;
  return h;
}

// kForSetup builds the per-sequence work list only (q, arena, out unused).
kvk_status prepare(const kvk_table* t, int32_t l0, int32_t l1, const void* q, int32_t q_dtype,
                   int32_t n_stored, float scale, const void* w_uk, const void* w_uv, const void* arena,
                   float* out, void* workspace, size_t ws_bytes, DecodePlan& P, PrepareMode mode = kForDecode) {
  if (!t) return fail(KVK_ERR_INVALID, "decode: NULL table");
  const kvk_dims& d = t->d;
  if (l0 < 0 || l1 > d.n_layers || l0 >= l1)
    return fail(KVK_ERR_INVALID, "layer range [%d, %d) invalid for %d layers", l0, l1, d.n_layers);
  if (mode == kForSetup) {
    q = arena = out = static_cast<float*>(workspace);
    q_dtype = KVK_BF16;
    n_stored = t->cap;
    scale = 1.0f;
  }
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
  const int32_t nl = l1 - l0;
  const bool batched = !t->seq.empty();
  const int32_t nbf_split = batched ? t->nb_cap : nbf;  // per-sequence lists: laid out for the capacity
  P.batched = batched;
  const ListLayout LL = batched ? list_layout(t, l0, l1) : ListLayout{0, 0, 0, 0};
  float* ws = reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) + LL.total);  // the partials
  DecodeArgs& a = P.d1;
  CombineArgs& ca = P.c1;
  a.arena = static_cast<const uint8_t*>(arena);
  a.q = q;
  a.ws = ws;
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
  a.items_dev = nullptr;
  a.list_hdr = nullptr;
  a.list_hash = 0;
  P.hash = 0;
  ca.out = out;
  ca.ws = ws;
  ca.arena = static_cast<const uint8_t*>(arena);
  ca.q = q;
  ca.q_f32 = q_dtype == KVK_F32;
  ca.scale_log2 = scale * kLog2e;
  ca.ntail = ntail;
  ca.nb_cap = t->nb_cap;
  ca.B = d.batch;
  ca.Hq = d.n_q_heads;
  ca.Hkv = d.n_kv_heads;
  ca.G = G;
  ca.n_layers = nl;
  ca.n_rows = nl * d.batch * d.n_q_heads;
  ca.citems = nullptr;
  ca.list_hdr = nullptr;
  ca.list_hash = 0;
  ca.nbf = nbf;
  ca.map = nullptr;

  const int64_t split_target = gqa_split_target(t, l0, l1);
  // One work item per distinct anchor read by the range (§2.1 depth sharing): per
  // anchor for all sequences, or per (sequence, anchor) under per-sequence plans.
  SmallVec<DecodeItem, kMaxItems> items;
  const int ngroups = batched ? d.batch : 1;
  SmallVec<int32_t, kMaxItems> l_item, l_slot;
  l_item.resize((size_t)ngroups * nl);
  l_slot.resize((size_t)ngroups * nl);
  int64_t ws_floats = 0;
  auto add_group = [&](const kvk_table* s, int g, int b0, int nb, int64_t base) {
    int item_of_anchor[KVK_MAX_LAYERS];
    for (int l = 0; l < KVK_MAX_LAYERS; ++l) item_of_anchor[l] = -1;
    for (int l = l0; l < l1; ++l) {
      const int anc = s->info.anchor_of[l];
      if (item_of_anchor[anc] < 0) {
        DecodeItem it;
        const int rb = anc > l0 ? anc : l0;
        const int re = s->next_anchor[anc] < l1 ? s->next_anchor[anc] : l1;
        it.region = base + s->info.layer_offset[anc];
        it.stream_bytes = (int32_t)s->info.stream_bytes[anc];
        it.block_bytes = (int32_t)s->block_bytes[anc];
        it.bits = s->bits[anc];
        it.q_layer0 = rb - l0;
        it.geff = G * (re - rb);
        it.split_blocks = gqa_item_split_blocks(s, anc, l0, l1, nbf_split, split_target);
        it.nsplit = n_splits(nbf_split, it.split_blocks);
        it.nchp = gqa_chunk_waves((it.geff + 15) / 16);
        it.b0 = b0;
        it.nb = nb;
        it.ws_off = (int32_t)ws_floats;
        ws_floats += (int64_t)nb * d.n_kv_heads * it.nsplit * it.geff * (D + 4);
        it.wave_begin = 0;
        item_of_anchor[anc] = (int)items.size();
        items.push_back(it);
      }
      const int ii = item_of_anchor[anc];
      l_item[(size_t)g * nl + (l - l0)] = ii;
      l_slot[(size_t)g * nl + (l - l0)] = (l - l0 - items[ii].q_layer0) * G;
    }
  };
  if (!batched) add_group(t, 0, 0, d.batch, 0);
  else
    for (int b = 0; b < d.batch; ++b) add_group(t->seq[b], b, b, 1, t->seq_base[b]);
  const int n_it = (int)items.size();

  // Launch order by precision: bf16, 2-bit, 8-bit, 4-bit.  The bf16 items (the
  // longest waves, bound by HBM) fill the GPU first; the 2-bit items (bound by their
  // unpacking) then run beside them rather than alone at the start or the end of the
  // launch.  Measured on the 14B mixed stack over all 24 orders (D1, one process):
  // this one 3258 us, 2/4/8/16 3346-3427 us, 16/8/4/2 3430 us, round-robin
  // interleaving of the items 3316-3380 us.  Item indices follow the new order;
  // wave_begin stays increasing.
  auto cost_rank = [](int bits) { return bits == 16 ? 0 : (bits == 2 ? 1 : (bits == 8 ? 2 : 3)); };
  SmallVec<int, kMaxItems> order, new_index;
  order.resize(n_it);
  new_index.resize(n_it);
  int n_ord = 0;
  for (int r = 0; r < 4; ++r)  // a stable counting sort by rank
    for (int k = 0; k < n_it; ++k)
      if (cost_rank(items[k].bits) == r) order[n_ord++] = k;
  SmallVec<DecodeItem, kMaxItems> sorted;
  sorted.resize(n_it);
  int64_t waves = 0;
  for (int k = 0; k < n_it; ++k) {
    DecodeItem it = items[order[k]];
    waves = (waves + 3) / 4 * 4;  // a chunk group never straddles a workgroup
    it.wave_begin = (int32_t)waves;
    int64_t units = (int64_t)it.nb * d.n_kv_heads * it.nsplit;
    if (it.nchp > 4) units = (units + 7) / 8 * 8;  // whole groups of 8 units (see the kernel)
    waves += units * it.nchp;
    sorted[k] = it;
    new_index[order[k]] = k;
  }
  if ((size_t)LL.total + (size_t)ws_floats * sizeof(float) > ws_bytes)
    return fail(KVK_ERR_BUFFER, "workspace %zu bytes < %lld needed", ws_bytes,
                (long long)(LL.total + ws_floats * (int64_t)sizeof(float)));
  if (ws_floats > 0x7fffffffLL) return fail(KVK_ERR_UNSUPPORTED, "workspace exceeds 2^31 floats");
  if (waves > 0x7ffffff0LL) return fail(KVK_ERR_UNSUPPORTED, "too many decode waves");
  a.n_items = n_it;
  a.total_waves = (int32_t)waves;
  if (!batched) {
    for (int k = 0; k < n_it; ++k) {
      const DecodeItem& it = sorted[k];
      a.items[k] = it;
      ca.item_ws_off[k] = it.ws_off;
      ca.item_nsplit[k] = it.nsplit;
      ca.item_geff[k] = it.geff;
      ca.item_tail[k] = it.region + (int64_t)t->nb_cap * it.block_bytes;
      ca.item_stream_bytes[k] = it.stream_bytes;
    }
    for (int l = 0; l < nl; ++l) {
      ca.layer_item[l] = new_index[l_item[l]];
      ca.layer_slot0[l] = l_slot[l];
    }
  } else {
    if ((int64_t)n_it * (int64_t)sizeof(DecodeItem) > LL.citems) return fail(KVK_ERR_DEVICE, "work list size");
    P.list.assign((size_t)LL.total, 0);
    DecodeItem* di = reinterpret_cast<DecodeItem*>(P.list.data() + LL.items);
    CombItem* ci = reinterpret_cast<CombItem*>(P.list.data() + LL.citems);
    int32_t* map = reinterpret_cast<int32_t*>(P.list.data() + LL.map);
    for (int k = 0; k < n_it; ++k) {
      const DecodeItem& it = sorted[k];
      di[k] = it;
      ci[k].tail = it.region + (int64_t)t->nb_cap * it.block_bytes;
      ci[k].ws_off = it.ws_off;
      ci[k].nsplit = it.nsplit;
      ci[k].geff = it.geff;
      ci[k].stream_bytes = it.stream_bytes;
      ci[k].b0 = it.b0;
      ci[k].split_blocks = it.split_blocks;
    }
    for (int l = 0; l < nl; ++l)
      for (int b = 0; b < d.batch; ++b) {
        map[((int64_t)l * d.batch + b) * 2] = new_index[l_item[(size_t)b * nl + l]];
        map[((int64_t)l * d.batch + b) * 2 + 1] = l_slot[(size_t)b * nl + l];
      }
    P.hash = fnv1a(P.list.data() + LL.items, (size_t)(LL.total - LL.items));
    uint64_t* hdr = reinterpret_cast<uint64_t*>(P.list.data() + LL.hdr);
    hdr[0] = kListMagic;
    hdr[1] = P.hash;
    uint8_t* wsb = static_cast<uint8_t*>(workspace);
    a.items_dev = reinterpret_cast<const DecodeItem*>(wsb + LL.items);
    a.list_hdr = reinterpret_cast<const uint64_t*>(wsb + LL.hdr);
    a.list_hash = P.hash;
    ca.citems = reinterpret_cast<const CombItem*>(wsb + LL.citems);
    ca.map = reinterpret_cast<const int32_t*>(wsb + LL.map);
    ca.list_hdr = a.list_hdr;
    ca.list_hash = P.hash;
    ca.nbf = nbf;
    if (mode == kForDecode) {
      bool ready = false;
      {
        std::lock_guard<std::mutex> lock(t->setup_mu);
        for (const kvk_table::DecodeSetup& s : t->setups)
          ready |= s.workspace == workspace && s.l0 == l0 && s.l1 == l1 && s.hash == P.hash;
      }
      if (!ready)
        return fail(KVK_ERR_INVALID,
                    "per-sequence plans: call kvk_decode_setup for layers [%d, %d) on this workspace first", l0, l1);
    }
  }
  P.qs = d.qscheme;
  P.head_dim = D;
  P.any_blocks = nbf > 0 && waves > 0;
  return check_gpu_buffers({q, arena, out, workspace}, "decode");
}

kvk_status launch_d1(const DecodePlan& P, hipStream_t st) {
  if (!P.any_blocks) return KVK_OK;
  const unsigned grid = (unsigned)((P.d1.total_waves + 3) / 4);
#define KVK_D1(DD, KK, BB) hipLaunchKernelGGL((gqa_decode_kernel<DD, KK, BB>), dim3(grid), dim3(256), 0, st, P.d1)
  if (P.head_dim == 128) {
    if (P.qs == KVK_Q_KIVI32) { if (P.batched) KVK_D1(128, kQsKivi, true); else KVK_D1(128, kQsKivi, false); }
    else if (P.qs == KVK_Q_GROUP64) { if (P.batched) KVK_D1(128, kQsG64, true); else KVK_D1(128, kQsG64, false); }
    else { if (P.batched) KVK_D1(128, kQsSym, true); else KVK_D1(128, kQsSym, false); }
  } else {
    if (P.qs == KVK_Q_KIVI32) { if (P.batched) KVK_D1(64, kQsKivi, true); else KVK_D1(64, kQsKivi, false); }
    else if (P.qs == KVK_Q_GROUP64) { if (P.batched) KVK_D1(64, kQsG64, true); else KVK_D1(64, kQsG64, false); }
    else { if (P.batched) KVK_D1(64, kQsSym, true); else KVK_D1(64, kQsSym, false); }
  }
#undef KVK_D1
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(KVK_ERR_DEVICE, "decode launch: %s", hipGetErrorString(e));
  return KVK_OK;
}

kvk_status launch_c1(const DecodePlan& P, hipStream_t st) {
  const unsigned grid = (unsigned)((P.c1.n_rows + 3) / 4);
  if (P.head_dim == 128) {
    if (P.batched) hipLaunchKernelGGL((gqa_combine_kernel<128, true>), dim3(grid), dim3(256), 0, st, P.c1);
    else hipLaunchKernelGGL((gqa_combine_kernel<128, false>), dim3(grid), dim3(256), 0, st, P.c1);
  } else {
    if (P.batched) hipLaunchKernelGGL((gqa_combine_kernel<64, true>), dim3(grid), dim3(256), 0, st, P.c1);
    else hipLaunchKernelGGL((gqa_combine_kernel<64, false>), dim3(grid), dim3(256), 0, st, P.c1);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(KVK_ERR_DEVICE, "combine launch: %s", hipGetErrorString(e));
  return KVK_OK;
}

// An MLA decode call that passes neither weight uses the table's attached ones
// (kvk_set_mla_weights), from the range's first layer on.
void mla_attached_weights(const kvk_table* t, int32_t l0, const void*& w_uk, const void*& w_uv) {
  const kvk_dims& d = t->d;
  if (d.kind != KVK_MLA || w_uk || w_uv || !t->mla_w_uk || l0 < 0 || l0 >= d.n_layers) return;
  w_uk = static_cast<const uint8_t*>(t->mla_w_uk) + (int64_t)l0 * d.n_q_heads * d.latent_dim * d.nope_dim * 2;
  w_uv = static_cast<const uint8_t*>(t->mla_w_uv) + (int64_t)l0 * d.n_q_heads * d.v_dim * d.latent_dim * 2;
}

// Argument checks shared by the MLA decode entry points.
kvk_status mla_check(const kvk_table* t, int32_t l0, int32_t l1, const void* q, int32_t q_dtype,
                     int32_t n_stored, float scale, const void* w_uk, const void* w_uv,
                     const void* arena, const void* out, const void* workspace, size_t ws_bytes) {
  const kvk_dims& d = t->d;
  if (l0 < 0 || l1 > d.n_layers || l0 >= l1)
    return fail(KVK_ERR_INVALID, "layer range [%d, %d) invalid for %d layers", l0, l1, d.n_layers);
  if (!q || !arena || !out || !workspace || !w_uk || !w_uv)
    return fail(KVK_ERR_INVALID, "NULL buffer (an MLA table needs q, w_uk, w_uv, arena, out, workspace)");
  if (q_dtype != KVK_BF16 && q_dtype != KVK_F32) return fail(KVK_ERR_INVALID, "q_dtype %d", q_dtype);
  if (n_stored < 0 || n_stored > t->cap)
    return fail(KVK_ERR_INVALID, "n_stored %d outside 0..%d", n_stored, t->cap);
  if (!(scale == scale)) return fail(KVK_ERR_INVALID, "scale is NaN");
  if ((reinterpret_cast<uintptr_t>(q) & 15) || (reinterpret_cast<uintptr_t>(arena) & 15) ||
      (reinterpret_cast<uintptr_t>(out) & 15) || (reinterpret_cast<uintptr_t>(w_uk) & 15) ||
      (reinterpret_cast<uintptr_t>(w_uv) & 15) || (reinterpret_cast<uintptr_t>(workspace) & 255))
    return fail(KVK_ERR_INVALID, "misaligned buffer (q/w_uk/w_uv/arena/out 16 B, workspace 256 B)");
  size_t need = 0;
  if (kvk_status st = kvk_workspace_bytes(t, l0, l1, &need)) return st;
  if (need > ws_bytes) return fail(KVK_ERR_BUFFER, "workspace %zu bytes < %zu needed", ws_bytes, need);
  return check_gpu_buffers({q, w_uk, w_uv, arena, out, workspace}, "decode");
}

}  // namespace

namespace kvk {
int64_t gqa_batched_list_bytes(const kvk_table* t, int32_t l0, int32_t l1) {
  return t->seq.empty() ? 0 : list_layout(t, l0, l1).total;
}
}  // namespace kvk

extern "C" kvk_status kvk_decode_attention(const kvk_table* t, int32_t l0, int32_t l1, const void* q,
                                           int32_t q_dtype, int32_t n_stored, float scale,
                                           const void* w_uk, const void* w_uv, const void* arena,
                                           float* out, void* workspace, size_t ws_bytes,
                                           hipStream_t stream) {
  if (t && t->d.kind == KVK_MLA) {
    mla_attached_weights(t, l0, w_uk, w_uv);
    kvk_status st = mla_check(t, l0, l1, q, q_dtype, n_stored, scale, w_uk, w_uv, arena, out, workspace,
                              ws_bytes);
    if (st != KVK_OK) return st;
    if (!t->seq.empty())
      return mla_decode_batched(t, l0, l1, q, q_dtype, n_stored, scale, w_uk, w_uv, arena, out, workspace,
                                stream, true, true);
    st = mla_decode_splits(t, l0, l1, q, q_dtype, n_stored, scale, w_uk, arena, workspace, stream);
    if (st != KVK_OK) return st;
    return mla_decode_merge(t, l0, l1, n_stored, w_uv, workspace, out, stream);
  }
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
  if (t && t->d.kind == KVK_MLA) {
    mla_attached_weights(t, l0, w_uk, w_uv);
    const kvk_status st = mla_check(t, l0, l1, q, q_dtype, n_stored, scale, w_uk, w_uv, arena, workspace,
                                    workspace, ws_bytes);
    if (st != KVK_OK) return st;
    if (!t->seq.empty())
      return mla_decode_batched(t, l0, l1, q, q_dtype, n_stored, scale, w_uk, w_uv, arena, nullptr, workspace,
                                stream, true, false);
    return mla_decode_splits(t, l0, l1, q, q_dtype, n_stored, scale, w_uk, arena, workspace, stream);
  }
  DecodePlan P;
  float* dummy_out = static_cast<float*>(workspace);  // not written by this phase
  kvk_status st = prepare(t, l0, l1, q, q_dtype, n_stored, scale, w_uk, w_uv, arena, dummy_out,
                          workspace, ws_bytes, P);
  if (st != KVK_OK) return st;
  return launch_d1(P, stream);
}

extern "C" kvk_status kvk_decode_merge(const kvk_table* t, int32_t l0, int32_t l1, const void* q,
                                       int32_t q_dtype, int32_t n_stored, float scale,
                                       const void* w_uk, const void* w_uv, const void* arena,
                                       const void* workspace, size_t ws_bytes, float* out,
                                       hipStream_t stream) {
  if (t && t->d.kind == KVK_MLA) {
    mla_attached_weights(t, l0, w_uk, w_uv);
    const kvk_status st = mla_check(t, l0, l1, q, q_dtype, n_stored, scale, w_uk, w_uv, arena, out,
                                    workspace, ws_bytes);
    if (st != KVK_OK) return st;
    if (!t->seq.empty())
      return mla_decode_batched(t, l0, l1, q, q_dtype, n_stored, scale, w_uk, w_uv, arena, out,
                                const_cast<void*>(workspace), stream, false, true);
    return mla_decode_merge(t, l0, l1, n_stored, w_uv, workspace, out, stream);
  }
  DecodePlan P;
  kvk_status st = prepare(t, l0, l1, q, q_dtype, n_stored, scale, w_uk, w_uv, arena, out,
                          const_cast<void*>(workspace), ws_bytes, P);
  if (st != KVK_OK) return st;
  return launch_c1(P, stream);
}

extern "C" kvk_status kvk_decode_setup(const kvk_table* t, int32_t l0, int32_t l1, void* workspace,
                                       size_t ws_bytes, hipStream_t stream) {
  if (!t) return fail(KVK_ERR_INVALID, "kvk_decode_setup: NULL table");
  if (l0 < 0 || l1 > t->d.n_layers || l0 >= l1)
    return fail(KVK_ERR_INVALID, "layer range [%d, %d) invalid for %d layers", l0, l1, t->d.n_layers);
  if (!workspace) return fail(KVK_ERR_INVALID, "kvk_decode_setup: NULL workspace");
  // one plan: the work list travels in the kernel arguments
  if (t->seq.empty()) return KVK_OK;
  DecodePlan P;
  MlaSeqList mla;
  if (t->d.kind == KVK_MLA) {
    MlaSeqList& L = mla;
    if (kvk_status st = mla_seq_list(t, l0, l1, L, true)) return st;
    size_t need = 0;
    if (kvk_status st = kvk_workspace_bytes(t, l0, l1, &need)) return st;
    if (need > ws_bytes) return fail(KVK_ERR_BUFFER, "workspace %zu bytes < %zu needed", ws_bytes, need);
    if (kvk_status st = check_gpu_buffers({workspace}, "kvk_decode_setup")) return st;
    P.list.swap(L.img);
    P.hash = L.hash;
  } else {
    kvk_status st = prepare(t, l0, l1, nullptr, KVK_BF16, 0, 1.0f, nullptr, nullptr, nullptr, nullptr, workspace,
                            ws_bytes, P, kForSetup);
    if (st != KVK_OK) return st;
  }
  {  // the workspace's earlier list (if any) is overwritten now
    std::lock_guard<std::mutex> lock(t->setup_mu);
    auto& v = t->setups;
    for (size_t i = 0; i < v.size();)
      if (v[i].workspace == workspace) v.erase(v.begin() + i);
      else ++i;
  }
  hipError_t e = hipMemcpyAsync(workspace, P.list.data(), P.list.size(), hipMemcpyHostToDevice, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);  // the host image is freed on return
  if (e != hipSuccess) return fail(KVK_ERR_DEVICE, "work list copy: %s", hipGetErrorString(e));
  kvk_table::DecodeSetup rec;
  rec.workspace = workspace;
  rec.l0 = l0;
  rec.l1 = l1;
  rec.hash = P.hash;
  if (t->d.kind == KVK_MLA) {
    rec.rows_off = mla.rows_off;
    rec.dmax = mla.dmax;
    for (int k = 0; k < 4; ++k) {
      rec.items_off[k] = mla.items_off[k];
      rec.n_items[k] = mla.n_items[k];
      rec.n_wg[k] = mla.n_wg[k];
    }
  }
  std::lock_guard<std::mutex> lock(t->setup_mu);
  t->setups.push_back(rec);
  return KVK_OK;
}

// ---------------------------------------------------------------------------
// The allocation-free decode entry point: kvk_decode_attention with the split
// partials (and, for MLA tables, the absorbed queries) in a file-scope device array
// instead of a caller workspace.  Each GPU holds its own copy of the array (from the
// first call on it until the process ends); its address on a device is looked up
// once, with that device current, and kept.  Nothing in the scratch needs clearing:
// every partial the merge reads is written by the split phase of the same call.
// ---------------------------------------------------------------------------
static __device__ __align__(256) uint8_t scratch[KVK_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

kvk_status scratch_on(hipStream_t stream, void** out) {
  int cur = 0;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess) return fail(KVK_ERR_DEVICE, "hipGetDevice: %s", hipGetErrorString(e));
  int dev = cur;
  if (stream) {
    e = hipStreamGetDevice(stream, &dev);
    if (e != hipSuccess) return fail(KVK_ERR_DEVICE, "hipStreamGetDevice: %s", hipGetErrorString(e));
  }
  if (dev < 0 || dev >= kMaxDevices) return fail(KVK_ERR_UNSUPPORTED, "device %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    if (dev != cur && (e = hipSetDevice(dev)) != hipSuccess)
      return fail(KVK_ERR_DEVICE, "hipSetDevice(%d): %s", dev, hipGetErrorString(e));
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (dev != cur) (void)hipSetDevice(cur);
    if (e != hipSuccess || !p)
      return fail(KVK_ERR_DEVICE, "scratch address on device %d: %s", dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return KVK_OK;
}

}  // namespace

extern "C" kvk_status kvk_decode_attention_noalloc(const kvk_table* t, int32_t l0, int32_t l1, const void* q,
                                                   int32_t q_dtype, int32_t n_stored, float scale,
                                                   const void* w_uk, const void* w_uv, const void* arena,
                                                   float* out, hipStream_t stream) {
  if (!t) return fail(KVK_ERR_INVALID, "decode: NULL table");
  if (!t->seq.empty())
    return fail(KVK_ERR_UNSUPPORTED, "the allocation-free decode takes one-plan tables only");
  size_t need = 0;
  kvk_status st = kvk_workspace_bytes(t, l0, l1, &need);
  if (st != KVK_OK) return st;
  if (need > (size_t)KVK_NOALLOC_SCRATCH_BYTES)
    return fail(KVK_ERR_UNSUPPORTED,
                "layers [%d, %d) need %zu bytes of scratch; the static scratch holds %zu: decode fewer "
                "layers per call",
                l0, l1, need, (size_t)KVK_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  st = scratch_on(stream, &ws);
  if (st != KVK_OK) return st;
  return kvk_decode_attention(t, l0, l1, q, q_dtype, n_stored, scale, w_uk, w_uv, arena, out, ws,
                              (size_t)KVK_NOALLOC_SCRATCH_BYTES, stream);
}

extern "C" kvk_status kvk_read_bytes(const kvk_table* t, int32_t l0, int32_t l1, int32_t n_stored,
                                     int64_t* out_bytes) {
  if (!t || !out_bytes) return fail(KVK_ERR_INVALID, "kvk_read_bytes: NULL argument");
  const kvk_dims& d = t->d;
  if (l0 < 0 || l1 > d.n_layers || l0 >= l1)
    return fail(KVK_ERR_INVALID, "layer range [%d, %d) invalid for %d layers", l0, l1, d.n_layers);
  if (n_stored < 0 || n_stored > t->cap)
    return fail(KVK_ERR_INVALID, "n_stored %d outside 0..%d", n_stored, t->cap);
  if (!t->seq.empty()) {  // per-sequence plans: each sequence's distinct anchors, once
    int64_t sum = 0;
    for (const kvk_table* s : t->seq) {
      int64_t one = 0;
      const kvk_status st = kvk_read_bytes(s, l0, l1, n_stored, &one);
      if (st != KVK_OK) return st;
      sum += one;
    }
    *out_bytes = sum;
    return KVK_OK;
  }
  bool seen[KVK_MAX_LAYERS] = {false};
  int64_t total = 0;
  const bool mla = d.kind == KVK_MLA;
  const int64_t streams = mla ? (int64_t)d.batch : (int64_t)d.batch * d.n_kv_heads;
  for (int l = l0; l < l1; ++l) {
    const int a = t->info.anchor_of[l];
    if (seen[a]) continue;
    seen[a] = true;
    // bf16 tail tokens: K and V of one head (GQA), or the d + d_R stored channels (MLA)
    const int64_t tail_tok = mla ? 2LL * (t->rank[a] + d.rope_dim) : 4LL * d.head_dim;
    const int64_t per = (int64_t)(n_stored / KVK_GROUP) * t->block_bytes[a] +
                        (int64_t)(n_stored % KVK_GROUP) * tail_tok;
    total += per * streams;
  }
  *out_bytes = total;
  return KVK_OK;
}
