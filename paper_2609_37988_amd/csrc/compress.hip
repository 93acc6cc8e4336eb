// Prefill write of a layer's compressed cache (W1), the decode-time append of one
// token (W3: a bf16 tail write, or on the 32nd token the quantisation of the
// completed group with W1's block quantiser), and the test-only dequantiser.
//
// An anchor layer stores, per (sequence, KV head), its keys and values — after an
// optional eviction gather (KV-Kaizen §3, long context: the evictor runs on the
// same cache and the ratios multiply) — quantised by the table's scheme
// (App. C.3: grouped asymmetric KIVI32, or the paper's symmetric per-row SYMROW),
// or as bf16 at b = 16 (§2.2: a b = 16 GQA layer is the uncompressed cache).
// The layout written is the one documented in include/kvk.h.
//
// One workgroup of 256 threads writes one 32-token block of one stream: it stages
// the block's K and V in LDS as fp32 (16-byte loads), computes the group metadata
// with several threads per group and lane reductions, then every thread assembles
// whole 32-bit words of codes so that the global stores are coalesced.  The kernel
// is specialised per head width, bit-width and scheme, so that the layout address
// arithmetic reduces to shifts and masks.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <vector>

#include "kvk_device.h"
#include "kvk_internal.h"

using namespace kvkd;

namespace {

// Sequences of a per-sequence batch one write launch serves (those whose plan gives
// the layer the same bit-width), and each one's region.
constexpr int kWriteSeqs = 64;

struct CompressArgs {
  const void* k;
  const void* v;
  const int32_t* keep;
  uint8_t* region;
  int64_t block_bytes;
  int64_t stream_bytes;
  int32_t in_f32;
  int32_t n_tokens;
  int32_t n_stored;
  int32_t nbf;      // full blocks written
  int32_t nb_cap;   // full-block capacity (tail block sits after it)
  int32_t D;
  int32_t bits;
  int32_t qs;       // kvk_qscheme
  // Per-sequence batches (n_seq > 0): the launch's streams are the Hkv streams of
  // sequences seq_of[0 .. n_seq), whose regions start seq_region[j] bytes after
  // `region`; the inputs stay indexed by the batch's sequence.  n_seq = 0: one table.
  int32_t n_seq, Hkv;
  int32_t seq_of[kWriteSeqs];
  int64_t seq_region[kWriteSeqs];
};

#pragma clang fp contract(off)

__device__ __forceinline__ uint32_t kivi_code(float x, float s, float z, float levels) {
  if (s == 0.0f) return 0u;
  const float t = (x - z) / s;  // IEEE fp32, correctly rounded
  const float r = fminf(fmaxf(rintf(t), 0.0f), levels);
  return (uint32_t)r;
}

__device__ __forceinline__ uint32_t sym_code(float x, float s, int bits) {
  const float q = (float)((1 << (bits - 1)) - 1);
  float r = 0.0f;
  if (s != 0.0f) r = fminf(fmaxf(rintf(x / s), -q), q);
  return (uint32_t)((int)r + (1 << (bits - 1)));
}

// Stage the 32 tokens of a block (K and V, fp32) in LDS: thread (token t, chunk q)
// moves channels 8q .. 8q+7 with 16-byte loads; tokens past ntok are zero.
template <int D, int LD>
__device__ __forceinline__ void stage_block(const CompressArgs& a, int stream, int tok0, int ntok, float* Ks,
                                            float* Vs, int tid) {
  constexpr int NQ = D / 8, TPP = 256 / NQ;  // chunks per row, tokens per pass
  const int q = tid % NQ;
  for (int t = tid / NQ; t < 32; t += TPP) {
    f4 k0 = {0.f, 0.f, 0.f, 0.f}, k1 = k0, v0 = k0, v1 = k0;
    if (t < ntok) {
      int pos = tok0 + t;
      if (a.keep) {
        pos = a.keep[(int64_t)stream * a.n_stored + pos];
        pos = pos < 0 ? 0 : (pos >= a.n_tokens ? a.n_tokens - 1 : pos);
      }
      const int64_t e = ((int64_t)stream * a.n_tokens + pos) * D + 8 * q;
      if (a.in_f32) {
        const f4* kp = reinterpret_cast<const f4*>(static_cast<const float*>(a.k) + e);
        const f4* vp = reinterpret_cast<const f4*>(static_cast<const float*>(a.v) + e);
        k0 = kp[0], k1 = kp[1], v0 = vp[0], v1 = vp[1];
      } else {
        const u4v kw = *reinterpret_cast<const u4v*>(static_cast<const uint16_t*>(a.k) + e);
        const u4v vw = *reinterpret_cast<const u4v*>(static_cast<const uint16_t*>(a.v) + e);
#pragma unroll
        for (int p = 0; p < 2; ++p) {
          k0[2 * p] = __uint_as_float(kw[p] << 16), k0[2 * p + 1] = __uint_as_float(kw[p] & 0xffff0000u);
          k1[2 * p] = __uint_as_float(kw[p + 2] << 16), k1[2 * p + 1] = __uint_as_float(kw[p + 2] & 0xffff0000u);
          v0[2 * p] = __uint_as_float(vw[p] << 16), v0[2 * p + 1] = __uint_as_float(vw[p] & 0xffff0000u);
          v1[2 * p] = __uint_as_float(vw[p + 2] << 16), v1[2 * p + 1] = __uint_as_float(vw[p + 2] & 0xffff0000u);
        }
      }
    }
    *reinterpret_cast<f4*>(&Ks[t * LD + 8 * q]) = k0;
    *reinterpret_cast<f4*>(&Ks[t * LD + 8 * q + 4]) = k1;
    *reinterpret_cast<f4*>(&Vs[t * LD + 8 * q]) = v0;
    *reinterpret_cast<f4*>(&Vs[t * LD + 8 * q + 4]) = v1;
  }
}

// bf16 block: 16-byte chunks of 8 values (see the bf16 block layout).
template <int D, int LD>
__device__ __forceinline__ void write_bf16_block(const float* Ks, const float* Vs, uint8_t* out, int tid) {
  uint4* o4 = reinterpret_cast<uint4*>(out);
  for (int ci = tid; ci < 8 * D; ci += 256) {
    uint32_t w[4];
    if (ci < 4 * D) {  // K tile tau: lane shares of D/2 bytes, dealt out in 16-byte pieces
      const int tau = ci / (2 * D), rem = ci % (2 * D);
      const int lam = rem & 63, j = rem >> 6;
      const int t = 16 * tau + (lam & 15), c0 = 32 * j + 8 * (lam >> 4);
#pragma unroll
      for (int p = 0; p < 4; ++p)
        w[p] = (uint32_t)f32_to_bf16_bits(Ks[t * LD + c0 + 2 * p]) |
               ((uint32_t)f32_to_bf16_bits(Ks[t * LD + c0 + 2 * p + 1]) << 16);
    } else {
      const int cv = ci - 4 * D;  // V: lane shares of D bytes
      const int lam = cv & 63, m = cv >> 6;
      const int c = 16 * m + (lam & 15), kg = lam >> 4;
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const int s0 = 2 * p, s1 = 2 * p + 1;
        const int t0 = 16 * (s0 >> 2) + 4 * kg + (s0 & 3), t1 = 16 * (s1 >> 2) + 4 * kg + (s1 & 3);
        w[p] = (uint32_t)f32_to_bf16_bits(Vs[t0 * LD + c]) | ((uint32_t)f32_to_bf16_bits(Vs[t1 * LD + c]) << 16);
      }
    }
    o4[ci] = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

// The inverse of write_bf16_block: a bf16 block (16-byte loads) into LDS rows as fp32.
template <int D, int LD>
__device__ __forceinline__ void stage_bf16_block(const uint8_t* in, float* Ks, float* Vs, int tid) {
  const uint4* i4 = reinterpret_cast<const uint4*>(in);
  for (int ci = tid; ci < 8 * D; ci += 256) {
    const uint4 q = i4[ci];
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
    if (ci < 4 * D) {
      const int tau = ci / (2 * D), rem = ci % (2 * D);
      const int lam = rem & 63, j = rem >> 6;
      const int t = 16 * tau + (lam & 15), c0 = 32 * j + 8 * (lam >> 4);
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        Ks[t * LD + c0 + 2 * p] = __uint_as_float(w[p] << 16);
        Ks[t * LD + c0 + 2 * p + 1] = __uint_as_float(w[p] & 0xffff0000u);
      }
    } else {
      const int cv = ci - 4 * D;
      const int lam = cv & 63, m = cv >> 6;
      const int c = 16 * m + (lam & 15), kg = lam >> 4;
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const int s0 = 2 * p, s1 = 2 * p + 1;
        const int t0 = 16 * (s0 >> 2) + 4 * kg + (s0 & 3), t1 = 16 * (s1 >> 2) + 4 * kg + (s1 & 3);
        Vs[t0 * LD + c] = __uint_as_float(w[p] << 16);
        Vs[t1 * LD + c] = __uint_as_float(w[p] & 0xffff0000u);
      }
    }
  }
}

// min / max over the N consecutive lanes of a group (N = 1, 2, 4), every lane of the
// group ending with the result.
template <int N>
__device__ __forceinline__ float group_min(float x) {
  if constexpr (N >= 2) x = fminf(x, dpp<kQuadXor1>(x));
  if constexpr (N >= 4) x = fminf(x, dpp<kQuadXor2>(x));
  return x;
}
template <int N>
__device__ __forceinline__ float group_max(float x) {
  if constexpr (N >= 2) x = fmaxf(x, dpp<kQuadXor1>(x));
  if constexpr (N >= 4) x = fmaxf(x, dpp<kQuadXor2>(x));
  return x;
}

// Quantise the 32 tokens staged in LDS (Ks, Vs: fp32 rows of LD floats) into one
// block of BITS-bit codes plus metadata at `out`.  Called by all 256 threads.
template <int D, int BITS, int QS>
__device__ __forceinline__ void write_quant_block(const float* Ks, const float* Vs, float* kmeta, float* vmeta,
                                                  uint8_t* out, int tid) {
  constexpr int LD = D + 4;
  {
    constexpr float levels = (float)((1 << BITS) - 1);

    // ---- group metadata ----
    constexpr int NG64 = D / 64;  // GROUP64 channel groups
    if constexpr (QS == kQsKivi) {
      {  // K: channel c over the block's 32 tokens, TPC threads per channel
        constexpr int TPC = 256 / D, TOK = 32 / TPC;
        const int c = tid / TPC, t0 = TOK * (tid % TPC);
        float mn = Ks[t0 * LD + c], mx = mn;
#pragma unroll
        for (int t = 1; t < TOK; ++t) {
          const float x = Ks[(t0 + t) * LD + c];
          mn = fminf(mn, x);
          mx = fmaxf(mx, x);
        }
        mn = group_min<TPC>(mn);
        mx = group_max<TPC>(mx);
        if (tid % TPC == 0) {
          kmeta[c] = (float)(_Float16)((mx - mn) / levels);
          kmeta[D + c] = (float)(_Float16)mn;
        }
      }
      {  // V: token t, channel group g (32 channels), TPG threads per group
        constexpr int NG = D / 32, TPG = 256 / (32 * NG), CH = 32 / TPG;
        const int pr = tid / TPG, t = pr / NG, g = pr % NG;
        const float* row = &Vs[t * LD + 32 * g + CH * (tid % TPG)];
        f4 x = *reinterpret_cast<const f4*>(row);
        float mn = fminf(fminf(x[0], x[1]), fminf(x[2], x[3])), mx = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
#pragma unroll
        for (int c = 4; c < CH; c += 4) {
          x = *reinterpret_cast<const f4*>(row + c);
          mn = fminf(mn, fminf(fminf(x[0], x[1]), fminf(x[2], x[3])));
          mx = fmaxf(mx, fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])));
        }
        mn = group_min<TPG>(mn);
        mx = group_max<TPG>(mx);
        if (tid % TPG == 0) {
          vmeta[2 * (t * NG + g)] = (float)(_Float16)((mx - mn) / levels);
          vmeta[2 * (t * NG + g) + 1] = (float)(_Float16)mn;
        }
      }
    } else if constexpr (QS == kQsG64) {  // (token, 64 channels) of K then of V, TPG threads per group
      constexpr int NGR = 2 * 32 * NG64, TPG = 256 / NGR, CH = 64 / TPG;
      const int pr = tid / TPG, isv = pr >= 32 * NG64, r = pr % (32 * NG64), t = r / NG64, g = r % NG64;
      const float* row = (isv ? &Vs[t * LD] : &Ks[t * LD]) + 64 * g + CH * (tid % TPG);
      f4 x = *reinterpret_cast<const f4*>(row);
      float mn = fminf(fminf(x[0], x[1]), fminf(x[2], x[3])), mx = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
#pragma unroll
      for (int c = 4; c < CH; c += 4) {
        x = *reinterpret_cast<const f4*>(row + c);
        mn = fminf(mn, fminf(fminf(x[0], x[1]), fminf(x[2], x[3])));
        mx = fmaxf(mx, fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])));
      }
      mn = group_min<TPG>(mn);
      mx = group_max<TPG>(mx);
      if (tid % TPG == 0) {
        float* meta = isv ? vmeta : kmeta;
        meta[2 * (t * NG64 + g)] = (float)(_Float16)((mx - mn) / levels);
        meta[2 * (t * NG64 + g) + 1] = (float)(_Float16)mn;
      }
    } else {  // SYMROW: one scale per token row of K (rows 0..31) and V (rows 32..63), 4 threads per row
      constexpr int CH = D / 4;
      const int r = tid >> 2;
      const float* row = (r < 32 ? &Ks[r * LD] : &Vs[(r - 32) * LD]) + CH * (tid & 3);
      float am = 0.0f;
#pragma unroll
      for (int c = 0; c < CH; c += 4) {
        const f4 x = *reinterpret_cast<const f4*>(row + c);
        am = fmaxf(am, fmaxf(fmaxf(fabsf(x[0]), fabsf(x[1])), fmaxf(fabsf(x[2]), fabsf(x[3]))));
      }
      am = group_max<4>(am);
      if ((tid & 3) == 0) {
        constexpr float q = (float)((1 << (BITS - 1)) - 1);
        const float sc = bf16_to_f32(f32_to_bf16_bits(am / q));
        if (r < 32) kmeta[r] = sc;
        else vmeta[r - 32] = sc;
      }
    }
    __syncthreads();

    // ---- codes: whole 32-bit words ----
    uint32_t* ow = reinterpret_cast<uint32_t*>(out);
    constexpr int cb = 4 * D * BITS;          // bytes per code region
    constexpr int lane_bytes_k = D * BITS / 32;
    constexpr int lane_bytes_v = D * BITS / 16;
    constexpr int nslot = 32 / BITS;          // codes per word
    for (int wi = tid; wi < 2 * cb / 4; wi += 256) {
      const bool isv = wi >= cb / 4;
      const int wb = 4 * (isv ? wi - cb / 4 : wi);  // byte offset inside the region
      int lam, r2, tau = 0;  // lane and byte of its share held by this word
      if (!isv) {
        tau = wb / (2 * D * BITS);
        share_of(lane_bytes_k, wb % (2 * D * BITS), lam, r2);
      } else {
        share_of(lane_bytes_v, wb, lam, r2);
      }
      const int i = lam & 15, kg = lam >> 4;
      // the chunk x and first slot s0 of the word's codes
      int x0, s0;
      if constexpr (BITS == 8) { x0 = r2 / 8; s0 = 4 * ((r2 % 8) / 4); }
      else if constexpr (BITS == 4) { x0 = r2 / 4; s0 = 0; }
      else { x0 = r2 / 2; s0 = 0; }
      uint32_t word = 0;
#pragma unroll
      for (int qq = 0; qq < nslot; ++qq) {
        int x, sl, bit;
        if constexpr (BITS == 8) { x = x0; sl = s0 + qq; bit = 8 * qq; }
        else if constexpr (BITS == 4) { x = x0; sl = qq; bit = 16 * (sl & 1) + 4 * (sl >> 1); }
        else { x = x0 + (qq >> 3); sl = qq & 7; bit = 16 * (sl & 1) + 2 * (sl >> 1) + 8 * (qq >> 3); }
        uint32_t u;
        if (!isv) {
          const int t = 16 * tau + i, c = 32 * x + 8 * kg + sl;
          const float xv = Ks[t * LD + c];
          if constexpr (QS == kQsKivi) {
            u = kivi_code(xv, kmeta[c], kmeta[D + c], levels);
          } else if constexpr (QS == kQsG64) {
            const int gi = 2 * (t * NG64 + (c >> 6));
            u = kivi_code(xv, kmeta[gi], kmeta[gi + 1], levels);
          } else {
            u = sym_code(xv, kmeta[t], BITS);
          }
        } else {
          const int c = 16 * x + i, t = 16 * (sl >> 2) + 4 * kg + (sl & 3);
          const float xv = Vs[t * LD + c];
          if constexpr (QS == kQsKivi) {
            const int g = c >> 5;
            u = kivi_code(xv, vmeta[2 * (t * (D / 32) + g)], vmeta[2 * (t * (D / 32) + g) + 1], levels);
          } else if constexpr (QS == kQsG64) {
            const int gi = 2 * (t * NG64 + (c >> 6));
            u = kivi_code(xv, vmeta[gi], vmeta[gi + 1], levels);
          } else {
            u = sym_code(xv, vmeta[t], BITS);
          }
        }
        word |= u << bit;
      }
      ow[wi] = word;
    }

    // ---- metadata stores ----
    uint16_t* om = reinterpret_cast<uint16_t*>(out + 2 * cb);
    if constexpr (QS == kQsG64) {
      for (int idx = tid; idx < 2 * D; idx += 256) {
        float val;
        if (idx < D) {  // K: ((tau*4 + kg)*NG*2 + g*2 + w)*4 + e, token 16 tau + 4 kg + e
          const int e = idx & 3, w = (idx >> 2) & 1, g = (idx >> 3) % NG64, tk = (idx >> 3) / NG64;
          const int t = 16 * (tk >> 2) + 4 * (tk & 3) + e;
          val = kmeta[2 * (t * NG64 + g) + w];
        } else {  // V: ((g*2 + w)*4 + kg)*8 + s, token 16 (s/4) + 4 kg + (s%4)
          const int e = idx - D;
          const int sl = e & 7, kg = (e >> 3) & 3, w = (e >> 5) & 1, g = e >> 6;
          const int t = 16 * (sl >> 2) + 4 * kg + (sl & 3);
          val = vmeta[2 * (t * NG64 + g) + w];
        }
        om[idx] = bitcast<uint16_t>((_Float16)val);  // exact: the value is an fp16
      }
    } else if constexpr (QS == kQsKivi) {
      for (int idx = tid; idx < 4 * D; idx += 256) {
        float val;
        if (idx < 2 * D) {
          val = kmeta[idx];  // scale[0..D) then zero[0..D)
        } else {
          const int e = idx - 2 * D;  // ((g*2 + w)*4 + kg)*8 + s
          const int sl = e & 7, kg = (e >> 3) & 3, w = (e >> 5) & 1, g = e >> 6;
          const int t = 16 * (sl >> 2) + 4 * kg + (sl & 3);
          val = vmeta[2 * (t * (D / 32) + g) + w];
        }
        om[idx] = bitcast<uint16_t>((_Float16)val);  // exact: the value is an fp16
      }
    } else if (tid < 64) {
      om[tid] = f32_to_bf16_bits(tid < 32 ? kmeta[tid] : vmeta[tid - 32]);
    }
  }
}

// One workgroup writes one 32-token block of one stream, with BITS-bit codes (or
// bf16 at BITS = 16; a stream's tail block is always bf16).
template <int D, int BITS, int QS>
__global__ __launch_bounds__(256) void compress_kernel(CompressArgs a) {
  constexpr int LD = D + 4;  // padded LDS row (floats), rows 16-byte aligned
  __shared__ float Ks[32 * LD];
  __shared__ float Vs[32 * LD];
  __shared__ float kmeta[2 * D];          // KIVI32: scale, zero per channel; GROUP64: per (token, group); SYMROW: row scale
  __shared__ float vmeta[2 * 32 * (D / 32)];

  const int tid = threadIdx.x;
  const int nblk = a.nbf + 1;
  const int stream = blockIdx.x / nblk;  // of the launch
  const int blk = blockIdx.x % nblk;
  const bool tail = blk == a.nbf;
  const int tok0 = blk * 32;
  const int ntok = tail ? a.n_stored - tok0 : 32;  // valid tokens of this block
  int in_stream = stream;                          // of the inputs
  uint8_t* sbase = a.region + (int64_t)stream * a.stream_bytes;
  if (a.n_seq > 0) {
    const int j = stream / a.Hkv, h = stream - j * a.Hkv;
    in_stream = a.seq_of[j] * a.Hkv + h;
    sbase = a.region + a.seq_region[j] + (int64_t)h * a.stream_bytes;
  }

  stage_block<D, LD>(a, in_stream, tok0, ntok, Ks, Vs, tid);
  __syncthreads();

  uint8_t* out = sbase + (tail ? (int64_t)a.nb_cap * a.block_bytes : (int64_t)blk * a.block_bytes);
  if (BITS == 16 || tail) {
    write_bf16_block<D, LD>(Ks, Vs, out, tid);
    return;
  }
  if constexpr (BITS != 16) write_quant_block<D, BITS, QS>(Ks, Vs, kmeta, vmeta, out, tid);
}

// Decode-time append of one token to every anchor of a layer range.
struct AppendItem {
  int64_t region;        // byte offset of the anchor's region (of one sequence's streams) in the arena
  int32_t stream_bytes;
  int32_t block_bytes;
  int32_t bits;
  int32_t row;           // the anchor's row in the new-token input (layer - layer_begin)
  int32_t s0;            // input stream (b * Hkv + kvh) of the item's first stream
  int32_t pad;
};

// Items per launch: kernel arguments are limited to 4 KiB.
constexpr int kAppendItems = 120;

struct AppendArgs {
  const void* k;         // [rows][B][Hkv][D] new keys
  const void* v;         // [rows][B][Hkv][D] new values
  uint8_t* arena;
  int32_t in_f32;
  int32_t pos;           // stored tokens before the call: the new token's position
  int32_t nb_cap;
  int32_t n_streams;     // streams per item: B * Hkv, or Hkv under per-sequence plans
  int64_t row_stride;    // elements between the rows of consecutive layers in k and v
  AppendItem items[kAppendItems];
};
static_assert(sizeof(AppendArgs) <= 4096, "kernel arguments");

__device__ __forceinline__ uint16_t new_token_bf16(const void* p, int64_t e, int in_f32) {
  return in_f32 ? f32_to_bf16_bits(static_cast<const float*>(p)[e]) : static_cast<const uint16_t*>(p)[e];
}

// The new token to slot pos % 32 of the bf16 tail block of every stream: one
// thread per (stream, channel), grid (streams * D / 256, anchors).
template <int D>
__global__ __launch_bounds__(256) void tail_write_kernel(AppendArgs a) {
  const int idx = blockIdx.x * 256 + threadIdx.x;
  if (idx >= a.n_streams * D) return;
  const int sidx = idx / D, c = idx % D, t = a.pos & 31;
  const AppendItem& it = a.items[blockIdx.y];
  uint8_t* tailb = a.arena + it.region + (int64_t)sidx * it.stream_bytes + (int64_t)a.nb_cap * it.block_bytes;
  const int64_t e = (int64_t)it.row * a.row_stride + (int64_t)(it.s0 + sidx) * D + c;
  *reinterpret_cast<uint16_t*>(tailb + k_bf16_byte(D, t, c)) = new_token_bf16(a.k, e, a.in_f32);
  *reinterpret_cast<uint16_t*>(tailb + v_bf16_byte(D, t, c)) = new_token_bf16(a.v, e, a.in_f32);
}

// The token that fills the tail (pos % 32 == 31) completes a 32-token group: one
// workgroup per (stream, anchor) quantises the tail's bf16 values plus the new
// token (rounded to bf16) into full block pos / 32, exactly as the prefill write
// quantises a block.  The tail is then empty (its stale slots are never read).
template <int D, int QS>
__global__ __launch_bounds__(256) void group_write_kernel(AppendArgs a) {
  constexpr int LD = D + 4;
  __shared__ float Ks[32 * LD];
  __shared__ float Vs[32 * LD];
  __shared__ float kmeta[2 * D];
  __shared__ float vmeta[2 * 32 * (D / 32)];
  const int tid = threadIdx.x, sidx = blockIdx.x;
  const AppendItem& it = a.items[blockIdx.y];
  uint8_t* base = a.arena + it.region + (int64_t)sidx * it.stream_bytes;
  uint8_t* tailb = base + (int64_t)a.nb_cap * it.block_bytes;
  const int64_t e0 = (int64_t)it.row * a.row_stride + (int64_t)(it.s0 + sidx) * D;
  stage_bf16_block<D, LD>(tailb, Ks, Vs, tid);  // row 31 holds a stale slot until replaced
  __syncthreads();
  for (int c = tid; c < D; c += 256) {
    Ks[31 * LD + c] = bf16_to_f32(new_token_bf16(a.k, e0 + c, a.in_f32));
    Vs[31 * LD + c] = bf16_to_f32(new_token_bf16(a.v, e0 + c, a.in_f32));
  }
  __syncthreads();
  uint8_t* out = base + (int64_t)(a.pos >> 5) * it.block_bytes;
  switch (it.bits) {
    case 16: write_bf16_block<D, LD>(Ks, Vs, out, tid); break;
    case 8: write_quant_block<D, 8, QS>(Ks, Vs, kmeta, vmeta, out, tid); break;
    case 4: write_quant_block<D, 4, QS>(Ks, Vs, kmeta, vmeta, out, tid); break;
    default: write_quant_block<D, 2, QS>(Ks, Vs, kmeta, vmeta, out, tid); break;
  }
}

// Test-only dequantiser: one thread per (stream, token, channel).
template <int D>
__global__ __launch_bounds__(256) void dequant_kernel(const uint8_t* region, int64_t stream_bytes,
                                                      int64_t block_bytes, int nb_cap, int n_stored,
                                                      int n_streams, int bits, int qs, float* kout,
                                                      float* vout) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t total = (int64_t)n_streams * n_stored * D;
  if (idx >= total) return;
  const int c = (int)(idx % D);
  const int64_t st = idx / D;
  const int tok = (int)(st % n_stored);
  const int stream = (int)(st / n_stored);
  const int blk = tok >> 5, t = tok & 31;
  const int nbf = n_stored >> 5;
  const uint8_t* base = region + (int64_t)stream * stream_bytes;
  float kv, vv;
  if (blk >= nbf || bits == 16) {
    const uint8_t* b = base + (blk >= nbf ? (int64_t)nb_cap * block_bytes : (int64_t)blk * block_bytes);
    kv = bf16_to_f32(*reinterpret_cast<const uint16_t*>(b + k_bf16_byte(D, t, c)));
    vv = bf16_to_f32(*reinterpret_cast<const uint16_t*>(b + v_bf16_byte(D, t, c)));
  } else {
    const uint8_t* b = base + (int64_t)blk * block_bytes;
    const uint32_t* w = reinterpret_cast<const uint32_t*>(b);
    const uint32_t mask = (1u << bits) - 1u;
    const int64_t kb = k_code_bit(D, bits, t, c), vb = v_code_bit(D, bits, t, c);
    const uint32_t uk = (w[kb >> 5] >> (kb & 31)) & mask;
    const uint32_t uv = (w[vb >> 5] >> (vb & 31)) & mask;
    const uint16_t* meta = reinterpret_cast<const uint16_t*>(b + 8LL * D * bits);
    if (qs == KVK_Q_GROUP64) {
      const int g = c >> 6, ng = D / 64;
      const int ki = (((t >> 4) * 4 + ((t >> 2) & 3)) * ng * 2 + g * 2) * 4 + (t & 3);
      kv = fmaf((float)uk, f16_bits_to_f32(meta[ki]), f16_bits_to_f32(meta[ki + 4]));
      vv = fmaf((float)uv, f16_bits_to_f32(meta[D + v_meta_index(t, g, 0)]),
                f16_bits_to_f32(meta[D + v_meta_index(t, g, 1)]));
    } else if (qs == KVK_Q_KIVI32) {
      kv = fmaf((float)uk, f16_bits_to_f32(meta[c]), f16_bits_to_f32(meta[D + c]));
      const int g = c >> 5;
      vv = fmaf((float)uv, f16_bits_to_f32(meta[2 * D + v_meta_index(t, g, 0)]),
                f16_bits_to_f32(meta[2 * D + v_meta_index(t, g, 1)]));
    } else {
      const int off = 1 << (bits - 1);
      kv = (float)((int)uk - off) * bf16_to_f32(meta[t]);
      vv = (float)((int)uv - off) * bf16_to_f32(meta[32 + t]);
    }
  }
  kout[idx] = kv;
  vout[idx] = vv;
}

}  // namespace

using namespace kvk;

// One W1 launch over `nstreams` streams of the arguments' layout.
static kvk_status launch_w1(const CompressArgs& a, int64_t nstreams, hipStream_t stream) {
  const int64_t grid = nstreams * (a.nbf + 1);
  if (grid > 0x7fffffffLL) return fail(KVK_ERR_UNSUPPORTED, "grid too large");
  const dim3 g3((unsigned)grid), b3(256);
#define KVK_W1(DD, BB, KK) \
  if (a.D == DD && a.bits == BB && (BB == 16 || a.qs == KK)) { \
    hipLaunchKernelGGL((compress_kernel<DD, BB, KK>), g3, b3, 0, stream, a); \
    launched = true; \
  }
  bool launched = false;
  KVK_W1(128, 16, 0) else KVK_W1(128, 8, 0) else KVK_W1(128, 4, 0) else KVK_W1(128, 2, 0)
  else KVK_W1(128, 8, 1) else KVK_W1(128, 4, 1) else KVK_W1(128, 2, 1)
  else KVK_W1(128, 8, 2) else KVK_W1(128, 4, 2) else KVK_W1(128, 2, 2)
  else KVK_W1(64, 16, 0) else KVK_W1(64, 8, 0) else KVK_W1(64, 4, 0) else KVK_W1(64, 2, 0)
  else KVK_W1(64, 8, 1) else KVK_W1(64, 4, 1) else KVK_W1(64, 2, 1)
  else KVK_W1(64, 8, 2) else KVK_W1(64, 4, 2) else KVK_W1(64, 2, 2)
#undef KVK_W1
  if (!launched) return fail(KVK_ERR_UNSUPPORTED, "no write kernel for d_h %d, %d bits", a.D, a.bits);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(KVK_ERR_DEVICE, "compress launch: %s", hipGetErrorString(e));
  return KVK_OK;
}

extern "C" kvk_status kvk_compress_layer(const kvk_table* t, int32_t layer, const void* k, const void* v,
                                         int32_t in_dtype, int32_t n_tokens, const int32_t* keep_idx,
                                         void* arena, hipStream_t stream) {
  if (!t) return fail(KVK_ERR_INVALID, "kvk_compress_layer: NULL table");
  const kvk_dims& d = t->d;
  if (layer < 0 || layer >= d.n_layers) return fail(KVK_ERR_INVALID, "layer %d out of range", layer);
  if (t->plan[layer].inherit) return KVK_OK;  // an inheriting layer writes nothing (§2.1)
  if (!k || !v || !arena) return fail(KVK_ERR_INVALID, "kvk_compress_layer: NULL buffer");
  if (in_dtype != KVK_BF16 && in_dtype != KVK_F32) return fail(KVK_ERR_INVALID, "in_dtype %d", in_dtype);
  if (n_tokens < 1 || n_tokens > d.max_tokens)
    return fail(KVK_ERR_INVALID, "n_tokens %d outside 1..max_tokens (%d)", n_tokens, d.max_tokens);
  const bool evict = d.keep_tokens > 0;
  if (evict && !keep_idx) return fail(KVK_ERR_INVALID, "the table evicts: keep_idx is required");
  if (!evict && keep_idx) return fail(KVK_ERR_INVALID, "the table does not evict: keep_idx must be NULL");
  if (evict && n_tokens < d.keep_tokens)
    return fail(KVK_ERR_INVALID, "n_tokens %d < keep_tokens %d", n_tokens, d.keep_tokens);
  if ((reinterpret_cast<uintptr_t>(arena) & 15) || (reinterpret_cast<uintptr_t>(k) & 15) ||
      (reinterpret_cast<uintptr_t>(v) & 15))
    return fail(KVK_ERR_INVALID, "misaligned buffer (16-byte alignment required)");
  if (kvk_status st = check_gpu_buffers({k, v, keep_idx, arena}, "kvk_compress_layer")) return st;
  if (!t->seq.empty()) {  // per-sequence plans: each sequence's own table and arena
    // The inputs stay indexed by the batch's sequence (GQA: K and V [B][Hkv][n][d_h];
    // MLA: latent [B][n][r] and positional key [B][n][d_R]).
    if (d.kind != KVK_MLA) {
      // One launch per bit-width for the sequences whose plans store the layer at it
      // (each sequence still written exactly as its one-sequence table writes it).
      for (const int bits : {16, 8, 4, 2}) {
        CompressArgs a;
        a.k = k;
        a.v = v;
        a.keep = keep_idx;
        a.region = static_cast<uint8_t*>(arena);
        a.in_f32 = in_dtype == KVK_F32;
        a.n_tokens = n_tokens;
        a.n_stored = evict ? d.keep_tokens : n_tokens;
        a.nbf = a.n_stored / KVK_GROUP;
        a.nb_cap = t->nb_cap;
        a.D = d.head_dim;
        a.bits = bits;
        a.qs = d.qscheme;
        a.Hkv = d.n_kv_heads;
        a.n_seq = 0;
        for (int b = 0; b < d.batch; ++b) {
          const kvk_table* s = t->seq[b];
          if (s->plan[layer].inherit || s->bits[layer] != bits) continue;
          a.block_bytes = s->block_bytes[layer];      // equal for every sequence at this bit-width
          a.stream_bytes = s->info.stream_bytes[layer];
          a.seq_of[a.n_seq] = b;
          a.seq_region[a.n_seq] = t->seq_base[b] + s->info.layer_offset[layer];
          if (++a.n_seq == kWriteSeqs) {
            const kvk_status st = launch_w1(a, (int64_t)a.n_seq * d.n_kv_heads, stream);
            if (st != KVK_OK) return st;
            a.n_seq = 0;
          }
        }
        if (a.n_seq > 0) {
          const kvk_status st = launch_w1(a, (int64_t)a.n_seq * d.n_kv_heads, stream);
          if (st != KVK_OK) return st;
        }
      }
      return KVK_OK;
    }
    return mla_compress_layer_batched(t, layer, k, v, in_dtype, n_tokens, keep_idx, arena, stream);
  }
  if (d.kind == KVK_MLA)
    return mla_compress_layer(t, layer, k, v, in_dtype, n_tokens, keep_idx, arena, stream);

  CompressArgs a;
  a.k = k;
  a.v = v;
  a.keep = keep_idx;
  a.region = static_cast<uint8_t*>(arena) + t->info.layer_offset[layer];
  a.block_bytes = t->block_bytes[layer];
  a.stream_bytes = t->info.stream_bytes[layer];
  a.in_f32 = in_dtype == KVK_F32;
  a.n_tokens = n_tokens;
  a.n_stored = evict ? d.keep_tokens : n_tokens;
  a.nbf = a.n_stored / KVK_GROUP;
  a.nb_cap = t->nb_cap;
  a.D = d.head_dim;
  a.bits = t->bits[layer];
  a.qs = d.qscheme;
  a.n_seq = 0;
  a.Hkv = d.n_kv_heads;
  return launch_w1(a, (int64_t)d.batch * d.n_kv_heads, stream);
}

static kvk_status append_gqa(const kvk_table* t, int32_t l0, int32_t l1, const void* k, const void* v,
                             int32_t in_dtype, int32_t n_stored, void* arena, hipStream_t stream);

extern "C" kvk_status kvk_compress_layer_project(const kvk_table* t, int32_t layer, const void* x,
                                                 const void* w_dkv, int32_t d_model, const void* k_rope,
                                                 int32_t n_tokens, const int32_t* keep_idx, void* arena,
                                                 void* latent_out, hipStream_t stream) {
  if (!t) return fail(KVK_ERR_INVALID, "kvk_compress_layer_project: NULL table");
  const kvk_dims& d = t->d;
  if (d.kind != KVK_MLA) return fail(KVK_ERR_INVALID, "kvk_compress_layer_project: an MLA table is required");
  if (layer < 0 || layer >= d.n_layers) return fail(KVK_ERR_INVALID, "layer %d out of range", layer);
  const bool per_seq = !t->seq.empty();
  if (per_seq && latent_out)
    return fail(KVK_ERR_INVALID, "kvk_compress_layer_project: latent_out must be NULL for per-sequence tables");
  if (!per_seq && t->plan[layer].inherit) return KVK_OK;  // an inheriting layer writes nothing (§2.1)
  if (!x || !w_dkv || !k_rope || !arena) return fail(KVK_ERR_INVALID, "kvk_compress_layer_project: NULL buffer");
  if (d_model < 32 || d_model % 32)
    return fail(KVK_ERR_INVALID, "d_model %d: a positive multiple of 32", d_model);
  if (n_tokens < 1 || n_tokens > d.max_tokens)
    return fail(KVK_ERR_INVALID, "n_tokens %d outside 1..max_tokens (%d)", n_tokens, d.max_tokens);
  const bool evict = d.keep_tokens > 0;
  if (evict && !keep_idx) return fail(KVK_ERR_INVALID, "the table evicts: keep_idx is required");
  if (!evict && keep_idx) return fail(KVK_ERR_INVALID, "the table does not evict: keep_idx must be NULL");
  if (evict && n_tokens < d.keep_tokens)
    return fail(KVK_ERR_INVALID, "n_tokens %d < keep_tokens %d", n_tokens, d.keep_tokens);
  if ((reinterpret_cast<uintptr_t>(arena) & 15) || (reinterpret_cast<uintptr_t>(x) & 15) ||
      (reinterpret_cast<uintptr_t>(w_dkv) & 15) || (reinterpret_cast<uintptr_t>(k_rope) & 15) ||
      (reinterpret_cast<uintptr_t>(latent_out) & 15))
    return fail(KVK_ERR_INVALID, "misaligned buffer (16-byte alignment required)");
  if (kvk_status st = check_gpu_buffers({x, w_dkv, k_rope, keep_idx, arena, latent_out}, "kvk_compress_layer_project"))
    return st;
  if (per_seq)  // each sequence's own table and arena, the inputs indexed by the batch's sequence
    return mla_compress_layer_project_batched(t, layer, x, w_dkv, d_model, k_rope, n_tokens, keep_idx, arena, stream);
  return mla_compress_layer_project(t, layer, x, w_dkv, d_model, k_rope, n_tokens, keep_idx, arena, latent_out,
                                    stream);
}

extern "C" kvk_status kvk_append_token(const kvk_table* t, int32_t l0, int32_t l1, const void* k, const void* v,
                                       int32_t in_dtype, int32_t n_stored, void* arena, hipStream_t stream) {
  if (!t) return fail(KVK_ERR_INVALID, "kvk_append_token: NULL table");
  const kvk_dims& d = t->d;
  if (l0 < 0 || l1 > d.n_layers || l0 >= l1)
    return fail(KVK_ERR_INVALID, "layer range [%d, %d) invalid for %d layers", l0, l1, d.n_layers);
  if (!k || !v || !arena) return fail(KVK_ERR_INVALID, "kvk_append_token: NULL buffer");
  if (in_dtype != KVK_BF16 && in_dtype != KVK_F32) return fail(KVK_ERR_INVALID, "in_dtype %d", in_dtype);
  if (n_stored < 0 || n_stored >= t->cap)
    return fail(KVK_ERR_INVALID, "n_stored %d: the stream holds at most %d tokens", n_stored, t->cap);
  if ((reinterpret_cast<uintptr_t>(arena) & 15) || (reinterpret_cast<uintptr_t>(k) & 15) ||
      (reinterpret_cast<uintptr_t>(v) & 15))
    return fail(KVK_ERR_INVALID, "misaligned buffer (16-byte alignment required)");
  bool stores = false;  // an anchor in the range (of some sequence's plan)
  for (size_t i = 0; i < (t->seq.empty() ? 1 : t->seq.size()); ++i)
    for (int l = l0; l < l1; ++l) stores |= !(t->seq.empty() ? t : t->seq[i])->plan[l].inherit;
  if (!stores) return KVK_OK;  // only inheritors: nothing is stored
  if (kvk_status st = check_gpu_buffers({k, v, arena}, "kvk_append_token")) return st;
  if (d.kind == KVK_MLA) return mla_append_token(t, l0, l1, k, v, in_dtype, n_stored, arena, stream);
  return append_gqa(t, l0, l1, k, v, in_dtype, n_stored, arena, stream);
}

// One item per (anchor layer) of a shared plan, over all B * Hkv streams; under
// per-sequence plans one per (sequence, anchor layer of its plan), over its Hkv
// streams.  Launched in groups of up to kAppendItems items.
static kvk_status append_gqa(const kvk_table* t, int32_t l0, int32_t l1, const void* k, const void* v,
                             int32_t in_dtype, int32_t n_stored, void* arena, hipStream_t stream) {
  const kvk_dims& d = t->d;
  const bool per_seq = !t->seq.empty();
  std::vector<AppendItem> items;
  for (int b = 0; b < (per_seq ? d.batch : 1); ++b) {
    const kvk_table* st = per_seq ? t->seq[b] : t;
    const int64_t base = per_seq ? t->seq_base[b] : 0;
    for (int l = l0; l < l1; ++l) {
      if (st->plan[l].inherit) continue;  // an inheriting layer stores nothing (§2.1)
      AppendItem it;
      it.region = base + st->info.layer_offset[l];
      it.stream_bytes = (int32_t)st->info.stream_bytes[l];
      it.block_bytes = (int32_t)st->block_bytes[l];
      it.bits = st->bits[l];
      it.row = l - l0;
      it.s0 = per_seq ? b * d.n_kv_heads : 0;
      it.pad = 0;
      items.push_back(it);
    }
  }
  AppendArgs a;
  a.k = k;
  a.v = v;
  a.arena = static_cast<uint8_t*>(arena);
  a.in_f32 = in_dtype == KVK_F32;
  a.pos = n_stored;
  a.nb_cap = t->nb_cap;
  a.n_streams = per_seq ? d.n_kv_heads : d.batch * d.n_kv_heads;
  a.row_stride = (int64_t)d.batch * d.n_kv_heads * d.head_dim;
  const int qs = d.qscheme;
  const dim3 b3(256);
  for (size_t i0 = 0; i0 < items.size(); i0 += kAppendItems) {
    const int n = (int)std::min<size_t>(kAppendItems, items.size() - i0);
    std::copy(items.begin() + i0, items.begin() + i0 + n, a.items);
    if (n_stored % KVK_GROUP != KVK_GROUP - 1) {
      const dim3 g3((unsigned)((a.n_streams * d.head_dim + 255) / 256), (unsigned)n);
      if (d.head_dim == 128) hipLaunchKernelGGL(tail_write_kernel<128>, g3, b3, 0, stream, a);
      else hipLaunchKernelGGL(tail_write_kernel<64>, g3, b3, 0, stream, a);
    } else {
      const dim3 g3((unsigned)a.n_streams, (unsigned)n);
      if (d.head_dim == 128) {
        if (qs == KVK_Q_KIVI32) hipLaunchKernelGGL((group_write_kernel<128, kQsKivi>), g3, b3, 0, stream, a);
        else if (qs == KVK_Q_GROUP64) hipLaunchKernelGGL((group_write_kernel<128, kQsG64>), g3, b3, 0, stream, a);
        else hipLaunchKernelGGL((group_write_kernel<128, kQsSym>), g3, b3, 0, stream, a);
      } else {
        if (qs == KVK_Q_KIVI32) hipLaunchKernelGGL((group_write_kernel<64, kQsKivi>), g3, b3, 0, stream, a);
        else if (qs == KVK_Q_GROUP64) hipLaunchKernelGGL((group_write_kernel<64, kQsG64>), g3, b3, 0, stream, a);
        else hipLaunchKernelGGL((group_write_kernel<64, kQsSym>), g3, b3, 0, stream, a);
      }
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(KVK_ERR_DEVICE, "append launch: %s", hipGetErrorString(e));
  }
  return KVK_OK;
}

extern "C" kvk_status kvk_debug_dequantize(const kvk_table* t, int32_t layer, int32_t n_stored,
                                           const void* arena, float* k_out, float* v_out,
                                           hipStream_t stream) {
  if (!t) return fail(KVK_ERR_INVALID, "kvk_debug_dequantize: NULL table");
  const kvk_dims& d = t->d;
  if (layer < 0 || layer >= d.n_layers) return fail(KVK_ERR_INVALID, "layer %d out of range", layer);
  if (!arena || !k_out || !v_out) return fail(KVK_ERR_INVALID, "NULL buffer");
  if (n_stored < 0 || n_stored > t->cap)
    return fail(KVK_ERR_INVALID, "n_stored %d outside 0..%d", n_stored, t->cap);
  if (n_stored == 0) return KVK_OK;
  if (kvk_status st = check_gpu_buffers({arena, k_out, v_out}, "kvk_debug_dequantize")) return st;
  if (d.kind == KVK_MLA && !t->seq.empty()) {
    // sequence b's values at b n_stored r (latent, rows of its own kept width) and
    // b n_stored d_R (positional key)
    for (int b = 0; b < d.batch; ++b) {
      const kvk_status st = mla_debug_dequantize(t->seq[b], layer, n_stored,
                                                 static_cast<const uint8_t*>(arena) + t->seq_base[b],
                                                 k_out + (int64_t)b * n_stored * d.latent_dim,
                                                 v_out + (int64_t)b * n_stored * d.rope_dim, stream);
      if (st != KVK_OK) return st;
    }
    return KVK_OK;
  }
  if (d.kind == KVK_MLA) return mla_debug_dequantize(t, layer, n_stored, arena, k_out, v_out, stream);
  if (!t->seq.empty()) {
    const int64_t per = (int64_t)d.n_kv_heads * n_stored * d.head_dim;
    for (int b = 0; b < d.batch; ++b) {
      const kvk_status st = kvk_debug_dequantize(t->seq[b], layer, n_stored,
                                                 static_cast<const uint8_t*>(arena) + t->seq_base[b],
                                                 k_out + b * per, v_out + b * per, stream);
      if (st != KVK_OK) return st;
    }
    return KVK_OK;
  }
  const int a = t->info.anchor_of[layer];
  const uint8_t* region = static_cast<const uint8_t*>(arena) + t->info.layer_offset[a];
  const int nstreams = d.batch * d.n_kv_heads;
  const int64_t total = (int64_t)nstreams * n_stored * d.head_dim;
  const int64_t grid = (total + 255) / 256;
  if (grid > 0x7fffffffLL) return fail(KVK_ERR_UNSUPPORTED, "grid too large");
  const int qs = d.qscheme;
  if (d.head_dim == 128)
    hipLaunchKernelGGL(dequant_kernel<128>, dim3((unsigned)grid), dim3(256), 0, stream, region,
                       t->info.stream_bytes[a], t->block_bytes[a], t->nb_cap, n_stored, nstreams,
                       t->bits[a], qs, k_out, v_out);
  else
    hipLaunchKernelGGL(dequant_kernel<64>, dim3((unsigned)grid), dim3(256), 0, stream, region,
                       t->info.stream_bytes[a], t->block_bytes[a], t->nb_cap, n_stored, nstreams,
                       t->bits[a], qs, k_out, v_out);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(KVK_ERR_DEVICE, "dequantise launch: %s", hipGetErrorString(e));
  return KVK_OK;
}
