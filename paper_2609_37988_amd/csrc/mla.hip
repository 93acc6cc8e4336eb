// The rank axis: MLA latent caches (KV-Kaizen §2.1 "Rank", App. C.2).
//
// An MLA layer stores per token the first d coordinates of its latent c (shared
// by every head) and the positional key k^R (d_R = 64, after RoPE), at b bits
// (App. C.3 quantisers: KIVI32 groups of 32 stored channels of one token, or the
// paper's symmetric scale per stored vector) or bf16.  Head h attends with query
// [q_nope ; q_rope] to keys [W_UK[h] c_t ; k^R_t] and values W_UV[h] c_t.  The
// content key takes no RoPE, so its projection moves onto the query (App. C.2):
//
//   q~_h = W_UK[h][:, :d]^T q_nope_h                    (A1: absorb, MFMA)
//   s_t  = scale (q~_h . c_t[:d] + q_rope_h . k^R_t)     (D2: MFMA, M = tokens,
//   o_lat = sum_t softmax(s)_t c_t[:d]                        N = heads, K = d + 64)
//   o_h  = W_UV[h][:, :d] o_lat                          (C2: merge + up-projection, MFMA)
//
// and the latent is read once per decode step for all heads: a dense contraction
// of the heads against the tokens, which is what the matrix cores are for.
//
// D2 work unit: one workgroup of 4 waves per (anchor, reader layer and head chunk,
// sequence, split); a chunk is two 16-head tiles (32 heads), the last one of a
// layer one tile when the padded head count is odd in tiles.  Per 32-token block
// the workgroup stages the block in LDS as fp16 (dequantised, or converted from
// bf16), then, per head tile of the chunk,
//   S^T[token, head] = C[token, :] . q~[head, :]   wave w: token tile w / KS, channel part w % KS
//   online softmax over the block                  8 threads per head
//   O^T[chan, head] += C^T[chan, token] P^T[token, head]   wave w: channel tiles w, w+4, ...
// Register ring: the next blocks' raw bytes are loaded while the current block
// is computed.  The absorbed query and the probabilities enter the MFMAs as
// fp16; accumulation is fp32.
//
// Writes: the prefill write (W2) and the decode-time append (W3) share one block
// writer that takes its rows from the input or from the stream's bf16 tail.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <type_traits>
#include <vector>

#include "kvk_device.h"
#include "kvk_internal.h"

using namespace kvkd;

namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kRope = 64;
constexpr int kMaxItems = 41;       // anchors per decode launch (kernel arguments <= 4 KiB)

typedef __amdgpu_buffer_rsrc_t Rsrc;

__device__ __forceinline__ Rsrc buffer_rsrc(const uint8_t* base, int nbytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(base), (short)0, nbytes, 0x00020000);
}

__device__ __forceinline__ f4 mfma16(half8 a, half8 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f4 mfmab(bf16x8 a, bf16x8 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float load_in(const void* p, int f32, int64_t i) {
  return f32 ? static_cast<const float*>(p)[i] : bf16_to_f32(static_cast<const uint16_t*>(p)[i]);
}

// Two bf16 values of a word -> fp16 pair (exact for values in the fp16 range).
__device__ __forceinline__ half2v bf16x2_to_half2(uint32_t w) {
  return h2(__uint_as_float(w << 16), __uint_as_float(w & 0xFFFF0000u));
}

__device__ __forceinline__ uint16_t bf16_bits_rne(float x) { return f32_to_bf16_bits(x); }

// ---------------------------------------------------------------------------
// W2: prefill write of one MLA layer
// ---------------------------------------------------------------------------

constexpr int kMlaWriteSeqs = 64;  // sequences of a per-sequence batch per write launch

struct MlaCompressArgs {
  const void* latent;  // [B][n_tokens][r]
  const void* rope;    // [B][n_tokens][64]
  const int32_t* keep; // [B][n_stored] or null
  uint8_t* region;
  int64_t stream_bytes;
  int64_t block_bytes;
  int32_t in_f32;
  int32_t n_tokens;
  int32_t n_stored;
  int32_t nbf;
  int32_t nb_cap;
  int32_t r;
  int32_t d;
  int32_t bits;
  int32_t kivi;
  // Per-sequence batches (n_seq > 0): launch row j writes sequence seq_of[j] (its
  // inputs indexed by the batch's sequence) into the stream seq_region[j] bytes after
  // `region`.  n_seq = 0: row b is sequence b of one table.
  int32_t n_seq;
  int32_t seq_of[kMlaWriteSeqs];
  int64_t seq_region[kMlaWriteSeqs];
};

__device__ __forceinline__ uint32_t kivi_code(float x, float s, float z, float levels) {
  if (s == 0.0f) return 0u;
  const float t = (x - z) / s;  // IEEE fp32, correctly rounded
  return (uint32_t)fminf(fmaxf(rintf(t), 0.0f), levels);
}

__device__ __forceinline__ uint32_t sym_code(float x, float s, int bits) {
  const float q = (float)((1 << (bits - 1)) - 1);
  float r = 0.0f;
  if (s != 0.0f) r = fminf(fmaxf(rintf(x / s), -q), q);
  return (uint32_t)((int)r + (1 << (bits - 1)));
}

// Slot n of a block (lane-ordered layout): token 16 T + i and the first of the 8
// channels 32 K + 8 g .. + 7, for n = (T NK + K) 64 + i + 16 g.
struct MlaSlot {
  int t, c;
};
__device__ __forceinline__ MlaSlot mla_slot(int n, int NK) {
  const int kq = n >> 6, T = kq / NK;
  return {16 * T + (n & 15), 32 * (kq - T * NK) + 8 * ((n >> 4) & 3)};
}

// The 8 stored channels c0 .. c0+7 of block row t (zeros past the stored tokens).
__device__ __forceinline__ void mla_load8(const MlaCompressArgs& a, int b, int tok0, int ntok, int t, int c0,
                                          float (&x)[8]) {
  if (t >= ntok) {
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = 0.0f;
    return;
  }
  int pos = tok0 + t;
  if (a.keep) {
    pos = a.keep[(int64_t)b * a.n_stored + pos];
    pos = pos < 0 ? 0 : (pos >= a.n_tokens ? a.n_tokens - 1 : pos);
  }
  const int64_t row = (int64_t)b * a.n_tokens + pos;
  const void* src = c0 < a.d ? a.latent : a.rope;
  const int64_t e0 = c0 < a.d ? row * a.r + c0 : row * kRope + (c0 - a.d);
  if (a.in_f32) {
    const f4* p = reinterpret_cast<const f4*>(static_cast<const float*>(src) + e0);
    const f4 lo = p[0], hi = p[1];
#pragma unroll
    for (int e = 0; e < 4; ++e) x[e] = lo[e], x[4 + e] = hi[e];
  } else {
    const u4v w = *reinterpret_cast<const u4v*>(static_cast<const uint16_t*>(src) + e0);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[2 * e] = __uint_as_float(w[e] << 16);
      x[2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
    }
  }
}

// The prefill source of a block: rows tok0 .. tok0 + 31 of sequence b of the input.
struct PrefillRows {
  const MlaCompressArgs& a;
  int b, tok0, ntok;
  __device__ __forceinline__ void load8(int t, int c0, float (&x)[8]) const { mla_load8(a, b, tok0, ntok, t, c0, x); }
};

// Write one 32-token block whose rows come from src.load8(t, c0, x) (the 8 stored
// channels c0 .. c0+7 of block row t).  Each wave takes (tile T, k-step K) tasks:
// lane (i, g) moves the 8 channels 32 K + 8 g .. + 7 of block row 16 T + i, i.e.
// exactly slot (T NK + K) 64 + i + 16 g, so loads and stores need no staging.
// KIVI32 groups (32 channels of one token) are the 4 lanes i, i + 16, i + 32, i + 48;
// SYMROW scales (one per token and vector) come from a first pass through LDS.
// Called by every thread of the workgroup (tid = threadIdx.x, nw waves); as_bf16
// writes the bf16 block instead.
template <int BITS, bool KIVI, class Src>
__device__ __forceinline__ void mla_write_block(const Src& src, uint8_t* out, int d, bool as_bf16,
                                                uint32_t (&amax)[2][32], int tid, int nw) {
#pragma clang fp contract(off)
  const int lane = tid & 63, wv = tid >> 6, i = lane & 15, g = lane >> 4;
  const int W = d + kRope, NK = W / 32;
  if (BITS == 16 || as_bf16) {  // bf16 block: 16 bytes (8 channels) per slot
    for (int task = wv; task < 2 * NK; task += nw) {
      const int T = task / NK, K = task - T * NK;
      float x[8];
      src.load8(16 * T + i, 32 * K + 8 * g, x);
      u4v o;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        o[e] = (uint32_t)bf16_bits_rne(x[2 * e]) | ((uint32_t)bf16_bits_rne(x[2 * e + 1]) << 16);
      *reinterpret_cast<u4v*>(out + 16 * ((T * NK + K) * 64 + i + 16 * g)) = o;
    }
    return;
  }
  if constexpr (BITS != 16) {
    constexpr float levels = (float)((1 << BITS) - 1);
    constexpr int cb_per_w = 4 * BITS;  // code bytes of the block per stored channel
    uint8_t* meta = out + cb_per_w * W;
    if constexpr (!KIVI) {
      if (tid < 64) amax[tid >> 5][tid & 31] = 0u;
      __syncthreads();
      for (int task = wv; task < 2 * NK; task += nw) {
        const int T = task / NK, K = task - T * NK;
        float x[8];
        src.load8(16 * T + i, 32 * K + 8 * g, x);
        float am = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) am = fmaxf(am, fabsf(x[e]));
        am = rows_max(am);
        if (g == 0) atomicMax(&amax[32 * K < d ? 0 : 1][16 * T + i], __float_as_uint(am));  // am >= 0
      }
      __syncthreads();
    }
    for (int task = wv; task < 2 * NK; task += nw) {
      const int T = task / NK, K = task - T * NK, t = 16 * T + i;
      float x[8];
      src.load8(t, 32 * K + 8 * g, x);
      uint32_t u[8];
      if constexpr (KIVI) {
        float mn = x[0], mx = x[0];
#pragma unroll
        for (int e = 1; e < 8; ++e) mn = fminf(mn, x[e]), mx = fmaxf(mx, x[e]);
        mn = rows_min(mn);
        mx = rows_max(mx);
        const _Float16 sh = (_Float16)((mx - mn) / levels);
        const _Float16 zh = (_Float16)mn;
        const float sc = (float)sh, zf = (float)zh;
#pragma unroll
        for (int e = 0; e < 8; ++e) u[e] = kivi_code(x[e], sc, zf, levels);
        if (g == 0)
          *reinterpret_cast<uint32_t*>(meta + 4 * ((T * NK + K) * 16 + i)) =
              (uint32_t)bitcast<uint16_t>(sh) | ((uint32_t)bitcast<uint16_t>(zh) << 16);
      } else {
        constexpr float q = (float)((1 << (BITS - 1)) - 1);
        const float sc = bf16_to_f32(bf16_bits_rne(__uint_as_float(amax[32 * K < d ? 0 : 1][t]) / q));
#pragma unroll
        for (int e = 0; e < 8; ++e) u[e] = sym_code(x[e], sc, BITS);
      }
      const int S = (T * NK + K) * 64 + i + 16 * g;
      if constexpr (BITS == 8) {
        uint32_t w0 = 0, w1 = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) w0 |= u[e] << (8 * e), w1 |= u[4 + e] << (8 * e);
        *reinterpret_cast<u2v*>(out + 8 * S) = u2v{w0, w1};
      } else if constexpr (BITS == 4) {
        uint32_t w = 0;
#pragma unroll
        for (int e = 0; e < 8; ++e) w |= u[e] << (16 * (e & 1) + 4 * (e >> 1));
        *reinterpret_cast<uint32_t*>(out + 4 * S) = w;
      } else {
        uint32_t w = 0;
#pragma unroll
        for (int e = 0; e < 8; ++e) w |= u[e] << (16 * (e & 1) + 2 * (e >> 1) + 8 * (g & 1));
        // sub-groups 2y and 2y + 1 (lanes 16 apart) share one word
        const auto sw = __builtin_amdgcn_permlane16_swap(w, w, false, false);
        w = sw[0] | sw[1];
        if ((g & 1) == 0) *reinterpret_cast<uint32_t*>(out + 4 * (((T * NK + K) * 16 + i) * 2 + (g >> 1))) = w;
      }
    }
    if constexpr (!KIVI) {
      if (tid < 64) {  // per token: the bf16 scale of c[:d] at byte 4t, of k^R at 4t + 2
        const int t = tid >> 1, part = tid & 1;
        constexpr float q = (float)((1 << (BITS - 1)) - 1);
        reinterpret_cast<uint16_t*>(meta)[tid] = bf16_bits_rne(__uint_as_float(amax[part][t]) / q);
      }
    }
  }
}

// One workgroup per (32-token block, sequence); a stream's tail block is bf16.
template <int BITS, bool KIVI>
__global__ __launch_bounds__(256) void mla_compress_kernel(MlaCompressArgs a) {
  __shared__ uint32_t amax[2][32];  // SYMROW: max |x| bits of (c[:d] | k^R, token)
  const int blk = blockIdx.x, j = blockIdx.y;
  const int b = a.n_seq > 0 ? a.seq_of[j] : j;
  const bool tail = blk == a.nbf;
  const int tok0 = 32 * blk;
  const PrefillRows src{a, b, tok0, tail ? a.n_stored - tok0 : 32};
  uint8_t* out = a.region + (a.n_seq > 0 ? a.seq_region[j] : (int64_t)j * a.stream_bytes) +
                 (tail ? (int64_t)a.nb_cap * a.block_bytes : (int64_t)blk * a.block_bytes);
  mla_write_block<BITS, KIVI>(src, out, a.d, tail, amax, threadIdx.x, 4);
}

// ---------------------------------------------------------------------------
// W2 with the down-projection (§2.1 "Rank", App. C.2): the latent's first d
// coordinates c[:d] = W_DKV[:d, :] x of each stored token on MFMA, rounded to bf16,
// then written by the block writer exactly as a latent input is.
// ---------------------------------------------------------------------------

struct MlaProjectArgs {
  const uint16_t* x;     // [B][n_tokens][H] bf16 hidden states
  const uint16_t* w;     // [r][H] bf16 W_DKV (row i -> latent coordinate i)
  const uint16_t* rope;  // [B][n_tokens][64] bf16 positional keys (after RoPE)
  const int32_t* keep;   // [B][n_stored] or null
  uint8_t* region;
  uint16_t* latent_out;  // [B][n_stored][d] bf16, or null
  int64_t stream_bytes;
  int64_t block_bytes;
  int32_t n_tokens;
  int32_t n_stored;
  int32_t nbf;
  int32_t nb_cap;
  int32_t H;
  int32_t d;
  // Per-sequence batches (n_seq > 0): launch row j writes sequence seq_of[j] (inputs
  // indexed by the batch's sequence) into the stream seq_region[j] bytes after
  // `region`; latent_out is then null.  n_seq = 0: row b is sequence b of one table.
  int32_t n_seq;
  int32_t seq_of[kMlaWriteSeqs];
  int64_t seq_region[kMlaWriteSeqs];
};

__device__ __forceinline__ int mla_stored_pos(const int32_t* keep, int b, int n_stored, int n_tokens, int pos) {
  if (!keep) return pos;
  const int p = keep[(int64_t)b * n_stored + pos];
  return p < 0 ? 0 : (p >= n_tokens ? n_tokens - 1 : p);
}

// The block writer's source for a projected block: the bf16 latent rows in LDS
// (pitch LP halfs) and the positional keys from the input.
struct ProjectedRows {
  const MlaProjectArgs& a;
  const uint16_t* lat;
  int LP, b, tok0, ntok;
  __device__ __forceinline__ void load8(int t, int c0, float (&x)[8]) const {
    if (t >= ntok) {
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = 0.0f;
      return;
    }
    u4v w;
    if (c0 < a.d) {
      w = *reinterpret_cast<const u4v*>(lat + t * LP + c0);
    } else {
      const int pos = mla_stored_pos(a.keep, b, a.n_stored, a.n_tokens, tok0 + t);
      w = *reinterpret_cast<const u4v*>(a.rope + ((int64_t)b * a.n_tokens + pos) * kRope + (c0 - a.d));
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[2 * e] = __uint_as_float(w[e] << 16);
      x[2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
    }
  }
};

// Geometry of the projected write for kept width D: TOK stored tokens per 8-wave
// workgroup (whole 32-token blocks); the waves split into WC channel groups x WT
// token groups, wave (wc, wt) owning CTW 16-channel tiles x TTW 16-token tiles of
// the latent tile.  Each k-step (32 of the model width) stages the W_DKV rows and
// the hidden-state rows in LDS (NBUF buffers, filled through registers one step
// ahead); the finished latent tile then takes the LDS as bf16 rows of pitch LP.
template <int D>
struct ProjGeo {
  static constexpr int TOK = D > 512 ? 64 : 128;
  static constexpr int NBLK = TOK / 32;
  static constexpr int CT = D / 16, TT = TOK / 16;
  static constexpr int WC = CT < 8 ? CT : 8, WT = 8 / WC;
  static constexpr int CTW = CT / WC, TTW = TT / WT;
  static constexpr int KP = 32 + 8;                   // staging row pitch (halfs): 16 rows, 16 bank windows
  static constexpr int NBUF = D > 512 ? 1 : 2;        // width 1024: one 85 KiB buffer
  static constexpr int NW = (4 * D + 511) / 512;      // 16-byte W_DKV chunks a thread stages per k-step
  static constexpr int LP = D + 8;                    // latent tile pitch (halfs)
  static constexpr int STAGE = NBUF * (D + TOK) * KP;
  static constexpr int LDS_HALFS = STAGE > TOK * LP ? STAGE : TOK * LP;
  static_assert(CT % WC == 0 && TT % WT == 0 && 4 * TOK <= 512, "tiles must split evenly over the waves");
};

// One 512-thread workgroup per (TOK stored tokens, sequence): the latent tile
// C[token][channel] = sum_k X[token][k] W[channel][k] on MFMA (A = W_DKV rows,
// B = hidden rows: a lane's accumulator holds 4 consecutive channels of one token),
// rounded to bf16 into LDS, then the tile's blocks (and the stream's tail block)
// written by the block writer with all 8 waves.
template <int D, int BITS, bool KIVI>
__global__ __launch_bounds__(512) void mla_project_kernel(MlaProjectArgs a) {
  using P = ProjGeo<D>;
  __shared__ __attribute__((aligned(16))) uint16_t lds[P::LDS_HALFS];
  __shared__ uint32_t amax[2][32];
  const int wg = blockIdx.x, j = blockIdx.y;
  const int b = a.n_seq > 0 ? a.seq_of[j] : j;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, i16 = lane & 15, kg = lane >> 4;
  const int wc = wv % P::WC, wt = wv / P::WC;
  const int row0 = P::TOK * wg;                         // first stored token of the tile
  const int nrow = min(P::TOK, a.n_stored - row0);      // may be <= 0 (the tail slot only)
  constexpr int BUF = (D + P::TOK) * P::KP;             // halfs per staging buffer: W rows, then hidden rows
  // W_DKV staging: chunk c = tid + 512 n < 4 D is row c / 4, k 8 (c % 4)
  const uint16_t* wsrc = a.w + (int64_t)(tid >> 2) * a.H + 8 * (tid & 3);
  const int64_t wstep = (int64_t)128 * a.H;             // 512 chunks = 128 rows further
  // hidden-row staging: thread tid < 4 TOK moves row tid / 4, k 8 (tid % 4)
  const int xr = tid >> 2, xk = 8 * (tid & 3);
  const bool x_stager = tid < 4 * P::TOK, x_ok = x_stager && xr < nrow;
  const uint16_t* xsrc = a.x + ((int64_t)b * a.n_tokens +
                                mla_stored_pos(a.keep, b, a.n_stored, a.n_tokens, x_ok ? row0 + xr : 0)) * a.H + xk;
  u4v wr[P::NW];
  auto fetch_w = [&](int k0) {
#pragma unroll
    for (int n = 0; n < P::NW; ++n)
      if (tid + 512 * n < 4 * D) wr[n] = *reinterpret_cast<const u4v*>(wsrc + n * wstep + k0);
  };
  auto store_w = [&](uint16_t* buf) {
#pragma unroll
    for (int n = 0; n < P::NW; ++n)
      if (tid + 512 * n < 4 * D)
        *reinterpret_cast<u4v*>(buf + (xr + 128 * n) * P::KP + xk) = wr[n];
  };
  auto fetch_x = [&](u4v& r, int k0) {
    r = x_ok ? *reinterpret_cast<const u4v*>(xsrc + k0) : u4v{0u, 0u, 0u, 0u};
  };
  auto store_x = [&](const u4v& r, uint16_t* buf) {
    if (x_stager) *reinterpret_cast<u4v*>(buf + (D + xr) * P::KP + xk) = r;
  };
  f4 acc[P::CTW][P::TTW];
#pragma unroll
  for (int j = 0; j < P::CTW; ++j)
#pragma unroll
    for (int m = 0; m < P::TTW; ++m) acc[j][m] = f4{0.f, 0.f, 0.f, 0.f};
  // the products of one k-step from a staging buffer
  auto step = [&](const uint16_t* base) {
    bf16x8 xb[P::TTW];
#pragma unroll
    for (int m = 0; m < P::TTW; ++m)
      xb[m] = *reinterpret_cast<const bf16x8*>(base + (D + 16 * (wt * P::TTW + m) + i16) * P::KP + 8 * kg);
#pragma unroll
    for (int j = 0; j < P::CTW; ++j) {
      const bf16x8 wa = *reinterpret_cast<const bf16x8*>(base + (16 * (wc * P::CTW + j) + i16) * P::KP + 8 * kg);
#pragma unroll
      for (int m = 0; m < P::TTW; ++m) acc[j][m] = mfmab(wa, xb[m], acc[j][m]);
    }
  };
  const int nks = a.H / 32;
  u4v xr0;
  fetch_w(0);
  fetch_x(xr0, 0);
  store_w(lds);
  store_x(xr0, lds);
  __syncthreads();
  for (int ks = 0; ks < nks; ++ks) {
    const int buf = P::NBUF == 2 ? (ks & 1) : 0;
    const bool more = ks + 1 < nks;  // uniform
    if (more) {
      fetch_w(32 * (ks + 1));
      fetch_x(xr0, 32 * (ks + 1));
    }
    step(lds + buf * BUF);
    if constexpr (P::NBUF == 2) {
      if (more) {  // the other buffer was last read before the previous barrier
        store_w(lds + (buf ^ 1) * BUF);
        store_x(xr0, lds + (buf ^ 1) * BUF);
      }
      __syncthreads();
    } else {
      __syncthreads();  // every wave is done with the buffer
      if (more) {
        store_w(lds);
        store_x(xr0, lds);
        __syncthreads();
      }
    }
  }
  // the latent tile, bf16, over the staging buffers (all reads of them are done)
#pragma unroll
  for (int j = 0; j < P::CTW; ++j) {
    const int c = 16 * (wc * P::CTW + j) + 4 * kg;
#pragma unroll
    for (int m = 0; m < P::TTW; ++m) {
      const int t = 16 * (wt * P::TTW + m) + i16;
      u2v w2;
      w2[0] = (uint32_t)f32_to_bf16_bits(acc[j][m][0]) | ((uint32_t)f32_to_bf16_bits(acc[j][m][1]) << 16);
      w2[1] = (uint32_t)f32_to_bf16_bits(acc[j][m][2]) | ((uint32_t)f32_to_bf16_bits(acc[j][m][3]) << 16);
      *reinterpret_cast<u2v*>(lds + t * P::LP + c) = w2;
      if (a.latent_out && t < nrow)
        *reinterpret_cast<u2v*>(a.latent_out + ((int64_t)b * a.n_stored + row0 + t) * a.d + c) = w2;
    }
  }
  __syncthreads();
  // block slots 0 .. nbf - 1 are full blocks, slot nbf the stream's bf16 tail block
  for (int k = 0; k < P::NBLK; ++k) {
    const int slot = P::NBLK * wg + k;  // uniform
    if (slot > a.nbf) break;
    const bool tail = slot == a.nbf;
    const ProjectedRows src_rows{a, lds + 32 * k * P::LP, P::LP, b, 32 * slot, tail ? a.n_stored - 32 * slot : 32};
    uint8_t* out = a.region + (a.n_seq > 0 ? a.seq_region[j] : (int64_t)j * a.stream_bytes) +
                   (tail ? (int64_t)a.nb_cap * a.block_bytes : (int64_t)slot * a.block_bytes);
    mla_write_block<BITS, KIVI>(src_rows, out, D, tail, amax, tid, 8);
    if constexpr (!KIVI) __syncthreads();  // amax is reused by the next block
  }
}

// Decode-time append of one token to every MLA anchor of a layer range.
struct MlaAppendItem {
  int64_t region;
  int32_t stream_bytes;
  int32_t block_bytes;
  int32_t bits;
  int32_t row;  // the anchor's row in the new-token input (layer - layer_begin)
  int32_t d;    // kept latent width
  int32_t seq;  // per-sequence plans: the one sequence (stream 0 of its region); -1: all
};

struct MlaAppendArgs {
  const void* latent;  // [rows][B][r] new latents
  const void* rope;    // [rows][B][d_R] new positional keys
  uint8_t* arena;
  int32_t in_f32;
  int32_t pos;         // stored tokens before the call: the new token's position
  int32_t nb_cap;
  int32_t B, r;
  MlaAppendItem items[KVK_MAX_LAYERS];
};

// The 8 stored channels c0 .. c0+7 of the new token, rounded to bf16 (the tail's
// precision), as fp32.
__device__ __forceinline__ void new_token8(const MlaAppendArgs& a, const MlaAppendItem& it, int b, int c0,
                                           float (&x)[8]) {
  const int64_t row = (int64_t)it.row * a.B + b;
  const void* src = c0 < it.d ? a.latent : a.rope;
  const int64_t e0 = c0 < it.d ? row * a.r + c0 : row * kRope + (c0 - it.d);
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const uint16_t hb = a.in_f32 ? bf16_bits_rne(static_cast<const float*>(src)[e0 + e])
                                 : static_cast<const uint16_t*>(src)[e0 + e];
    x[e] = bf16_to_f32(hb);
  }
}

__device__ __forceinline__ int mla_slot_of(int t, int c0, int NK) {
  return ((t >> 4) * NK + (c0 >> 5)) * 64 + (t & 15) + 16 * ((c0 >> 3) & 3);
}

// The rows of a completed group: tail slots 0..30 and the new token as row 31.
struct TailRows {
  const MlaAppendArgs& a;
  const MlaAppendItem& it;
  const uint8_t* tail;
  int b, NK;
  __device__ __forceinline__ void load8(int t, int c0, float (&x)[8]) const {
    if (t == 31) {
      new_token8(a, it, b, c0, x);
      return;
    }
    const u4v w = *reinterpret_cast<const u4v*>(tail + 16 * mla_slot_of(t, c0, NK));
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[2 * e] = __uint_as_float(w[e] << 16);
      x[2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
    }
  }
};

// One workgroup per (anchor, sequence): the token goes to slot pos % 32 of the bf16
// tail; the token that fills the tail completes a 32-token group, written as full
// block pos / 32 from the tail's bf16 rows exactly as the prefill write does.
template <bool KIVI>
__global__ __launch_bounds__(256) void mla_append_kernel(MlaAppendArgs a) {
  __shared__ uint32_t amax[2][32];
  const MlaAppendItem& it = a.items[blockIdx.y];
  const int b = it.seq >= 0 ? it.seq : blockIdx.x;  // the input row's sequence
  const int W = it.d + kRope, NK = W / 32, t = a.pos & 31;
  uint8_t* base = a.arena + it.region + (it.seq >= 0 ? 0 : (int64_t)b * it.stream_bytes);
  uint8_t* tail = base + (int64_t)a.nb_cap * it.block_bytes;
  if (t != 31) {
    for (int ch = threadIdx.x; ch < W / 8; ch += 256) {
      float x[8];
      new_token8(a, it, b, 8 * ch, x);
      u4v o;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        o[e] = (uint32_t)bf16_bits_rne(x[2 * e]) | ((uint32_t)bf16_bits_rne(x[2 * e + 1]) << 16);
      *reinterpret_cast<u4v*>(tail + 16 * mla_slot_of(t, 8 * ch, NK)) = o;
    }
    return;
  }
  const TailRows src{a, it, tail, b, NK};
  uint8_t* out = base + (int64_t)(a.pos >> 5) * it.block_bytes;
  switch (it.bits) {
    case 16: mla_write_block<16, KIVI>(src, out, it.d, true, amax, threadIdx.x, 4); break;
    case 8: mla_write_block<8, KIVI>(src, out, it.d, false, amax, threadIdx.x, 4); break;
    case 4: mla_write_block<4, KIVI>(src, out, it.d, false, amax, threadIdx.x, 4); break;
    default: mla_write_block<2, KIVI>(src, out, it.d, false, amax, threadIdx.x, 4); break;
  }
}

// Test-only dequantiser: one thread per (sequence, token, stored channel).
__global__ __launch_bounds__(256) void mla_dequant_kernel(const uint8_t* region, int64_t stream_bytes,
                                                          int64_t block_bytes, int nb_cap, int n_stored,
                                                          int B, int d, int bits, int kivi, float* cout,
                                                          float* rout) {
  const int W = d + kRope;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)B * n_stored * W) return;
  const int c = (int)(idx % W);
  const int64_t bt = idx / W;
  const int tok = (int)(bt % n_stored);
  const int b = (int)(bt / n_stored);
  const int blk = tok >> 5, t = tok & 31;
  const int nbf = n_stored >> 5;
  const uint8_t* base = region + (int64_t)b * stream_bytes;
  float x;
  const int NK = W / 32, T = t >> 4, i = t & 15, K = c >> 5, g = (c >> 3) & 3, s = c & 7;
  const int slot = (T * NK + K) * 64 + i + 16 * g;
  if (blk >= nbf || bits == 16) {
    const uint8_t* bb = base + (blk >= nbf ? (int64_t)nb_cap * block_bytes : (int64_t)blk * block_bytes);
    x = bf16_to_f32(*reinterpret_cast<const uint16_t*>(bb + 16 * slot + 2 * s));
  } else {
    const uint8_t* bb = base + (int64_t)blk * block_bytes;
    int wi, bit;
    if (bits == 8) {
      wi = 2 * slot + (s >> 2), bit = 8 * (s & 3);
    } else if (bits == 4) {
      wi = slot, bit = 16 * (s & 1) + 4 * (s >> 1);
    } else {
      wi = ((T * NK + K) * 16 + i) * 2 + (g >> 1), bit = 16 * (s & 1) + 2 * (s >> 1) + 8 * (g & 1);
    }
    const uint32_t u = (reinterpret_cast<const uint32_t*>(bb)[wi] >> bit) & ((1u << bits) - 1u);
    const uint16_t* meta = reinterpret_cast<const uint16_t*>(bb + 4 * W * bits);
    if (kivi) {
      const int p = (T * NK + K) * 16 + i;
      x = fmaf((float)u, f16_bits_to_f32(meta[2 * p]), f16_bits_to_f32(meta[2 * p + 1]));
    } else {
      x = (float)((int)u - (1 << (bits - 1))) * bf16_to_f32(meta[2 * t + (c >= d ? 1 : 0)]);
    }
  }
  if (c < d) cout[bt * d + c] = x;
  else rout[bt * kRope + (c - d)] = x;
}

// A per-sequence table's work list sits at the head of the workspace: this header,
// then its rows and items, hashed, so that a kernel reading a list that is not its
// call's returns without touching memory through it.
constexpr uint64_t kMlaListMagic = 0x4b564b4d4c413031ull;  // "KVKMLA01"

// One (layer of the range, sequence) of a per-sequence table: where its absorbed
// queries and split partials sit in the workspace, its kept width and split rule.
struct MlaSeqRow {
  int64_t q_off;         // fp16 [Hp][d + 64]
  int64_t part_off;      // fp32 [units_cap][Hp][d + 2]
  int32_t d;
  int32_t units_cap;
  int32_t split_target, split_nr;
};
static_assert(sizeof(MlaSeqRow) == 32, "MlaSeqRow without padding");

__device__ __forceinline__ bool mla_list_ok(const uint64_t* hdr, uint64_t hash) {
  return !hdr || (hdr[0] == kMlaListMagic && hdr[1] == hash);
}

// ---------------------------------------------------------------------------
// A1: absorbed queries, q~ = W_UK[h][:, :d]^T q_nope (scaled into the exp2 domain)
// ---------------------------------------------------------------------------

struct MlaAbsorbArgs {
  const void* q;          // [nl][B][Hq][nope + 64]
  const uint16_t* w_ukt;  // [nl][Hq][r][nope] bf16: W_UK[h] transposed (latent-major)
  uint8_t* ws;
  int64_t q_off[KVK_MAX_LAYERS];  // per relative layer: fp16 [B][Hp][d + 64]
  int32_t d_of[KVK_MAX_LAYERS];
  const MlaSeqRow* rows;  // per-sequence tables: per (relative layer, sequence) (else NULL)
  const uint64_t* list_hdr;
  uint64_t list_hash;
  int32_t q_f32;
  int32_t B, Hq, Hp, nope, r;  // Hp: Hq rounded up to whole 16-head tiles
  int64_t q_lstride;           // elements between consecutive layers' queries
  float scale_log2;
};

// Where sequence b's absorbed queries of relative layer li go, and their kept width:
// one plan, [B][Hp][d + 64] at q_off[li]; per-sequence plans, [Hp][d_b + 64] at the
// sequence's row.
__device__ __forceinline__ _Float16* absorb_dst(const MlaAbsorbArgs& a, int li, int b, int& d) {
  if (a.rows) {
    const MlaSeqRow& rw = a.rows[(int64_t)li * a.B + b];
    d = rw.d;
    return reinterpret_cast<_Float16*>(a.ws + rw.q_off);
  }
  d = a.d_of[li];
  return reinterpret_cast<_Float16*>(a.ws + a.q_off[li]) + (int64_t)b * a.Hp * (d + kRope);
}

// One workgroup per (layer, head, 16 sequences).  The 16 queries are staged in LDS
// and split into bf16 hi + lo B operands (K = nope); wave w then runs the 16-channel
// tiles w, w + 4, ... of the latent: A = rows of W_UK[h]^T (latent channel x nope,
// contiguous in the latent-major layout), up to the widest kept width of the 16
// (per-sequence plans: each sequence keeps the channels below its own).
__global__ __launch_bounds__(256) void mla_absorb_kernel(MlaAbsorbArgs a) {
  constexpr int PQ = 256 + 8;  // LDS row pitch of the queries (floats)
  __shared__ float qs[16 * PQ];
  if (!mla_list_ok(a.list_hdr, a.list_hash)) return;  // not this call's list
  const int li = blockIdx.x, h = blockIdx.y, b0 = 16 * blockIdx.z;
  const int nb = min(16, a.B - b0);
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, g = lane >> 4, i16 = lane & 15;
  const int qw = a.nope + kRope;
  const int nks = a.nope / 32;
  if (h >= a.Hq) {  // a padding head: zero query (finite scores, never written out)
    const int wmax = a.r + kRope;
    for (int e = tid; e < nb * wmax; e += 256) {
      const int bi = e / wmax, c = e - bi * wmax;
      int d;
      _Float16* qa = absorb_dst(a, li, b0 + bi, d);
      if (c < d + kRope) qa[(int64_t)h * (d + kRope) + c] = (_Float16)0.0f;
    }
    return;
  }
  for (int e = tid; e < nb * kRope; e += 256) {  // the RoPE part, scaled
    const int bi = e / kRope, j = e - bi * kRope;
    int d;
    _Float16* qa = absorb_dst(a, li, b0 + bi, d);
    const float x = load_in(a.q, a.q_f32, li * a.q_lstride + ((int64_t)(b0 + bi) * a.Hq + h) * qw + a.nope + j);
    qa[(int64_t)h * (d + kRope) + d + j] = (_Float16)(x * a.scale_log2);
  }
  const uint16_t* wt = a.w_ukt + ((int64_t)li * a.Hq + h) * a.r * a.nope;
  int d = 0;  // the widest kept width of the 16 sequences
#pragma unroll
  for (int bi = 0; bi < 16; ++bi) {
    if (bi < nb) {
      int db;
      absorb_dst(a, li, b0 + bi, db);
      d = db > d ? db : d;
    }
  }
  for (int e = tid; e < 16 * a.nope; e += 256) {
    const int bi = e / a.nope, i = e - bi * a.nope;
    qs[bi * PQ + i] = bi < nb ? load_in(a.q, a.q_f32, li * a.q_lstride + ((int64_t)(b0 + bi) * a.Hq + h) * qw + i) : 0.0f;
  }
  __syncthreads();
  bf16x8 bh[8], bl[8];  // nope <= 256
#pragma unroll
  for (int ks = 0; ks < 8; ++ks) {
    if (ks < nks) {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float x = qs[i16 * PQ + 32 * ks + 8 * g + j];
        const uint16_t hb = bf16_bits_rne(x);
        bh[ks][j] = bitcast<__bf16>(hb);
        bl[ks][j] = bitcast<__bf16>(bf16_bits_rne(x - bf16_to_f32(hb)));
      }
    }
  }
  const int bq = b0 + i16;
  int dq = 0;
  _Float16* qa = i16 < nb ? absorb_dst(a, li, bq, dq) : nullptr;
  for (int c = 16 * wv; c < d; c += 64) {
    const uint16_t* wrow = wt + (int64_t)(c + i16) * a.nope + 8 * g;
    u4v wa[8];
#pragma unroll
    for (int ks = 0; ks < 8; ++ks)
      if (ks < nks) wa[ks] = *reinterpret_cast<const u4v*>(wrow + 32 * ks);
    f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      if (ks < nks) {
        acc = mfmab(bitcast<bf16x8>(wa[ks]), bh[ks], acc);
        acc = mfmab(bitcast<bf16x8>(wa[ks]), bl[ks], acc);
      }
    }
    // D[chan c + 4g + e][seq i16]; kept widths are multiples of 32: a tile is wholly in or out
    if (i16 < nb && c < dq) {
      _Float16* dst = qa + (int64_t)h * (dq + kRope) + c + 4 * g;
#pragma unroll
      for (int e = 0; e < 4; ++e) dst[e] = (_Float16)(acc[e] * a.scale_log2);
    }
  }
}

// ---------------------------------------------------------------------------
// D2: decode over the stored latent
// ---------------------------------------------------------------------------

struct MlaItem {
  int64_t region;       // anchor's region in the arena
  int64_t q_off0;       // absorbed queries of the first reader layer
  int64_t q_stride;     // ... and between consecutive readers
  int64_t part_off0;    // split partials of the first reader layer
  int64_t part_stride;
  int32_t stream_bytes;
  int32_t block_bytes;
  int32_t d;
  int32_t bits;
  int32_t nreaders;     // reader layers (consecutive)
  int32_t nhc;          // head chunks per layer (32 heads; the last may hold 16)
  int32_t units;        // splits per stream the item's workgroups are laid out for
  int32_t units_cap;    // partial records per stream
  int32_t split_blocks;
  int32_t wg_begin;
  int32_t nseq;         // sequences (streams) of the item
  // Per-sequence items (written once, before the stored length is known): the split
  // rule (mla_split_len), from which the kernel takes the split length and the
  // splits of the call; split_nr = 0: split_blocks and units hold them.
  int32_t split_target, split_nr;
  int32_t reserved;     // (zero: the struct has no padding, and lists hash byte for byte)
};
static_assert(sizeof(MlaItem) == 96, "MlaItem without padding");

struct MlaDecodeArgs {
  const uint8_t* arena;
  uint8_t* ws;
  MlaItem items[kMaxItems];
  const MlaItem* items_dev;  // per-sequence tables: the items in the workspace (else NULL)
  const uint64_t* list_hdr;  // ... and the list's header, with the hash it must carry
  uint64_t list_hash;
  int32_t n_items;
  int32_t n_wg;
  int32_t B, Hq;         // Hq: the padded head count (whole 16-head tiles)
  int32_t nbf;          // full blocks per stream
  int32_t ntail;        // tail tokens
  int32_t nb_cap;
};
static_assert(sizeof(MlaDecodeArgs) <= 4096, "kernel arguments");


constexpr int kWaves = 4;  // waves per D2 workgroup (two workgroups share a CU)

// Geometry of the D2 workgroup for a kept width D (W = D + 64 stored channels).
// Wave w takes the 16 tokens of tile w / KS of the iteration and the channel part
// w % KS of them (KS = 2 for the widest rows, whose query for both head tiles would
// not fit the registers otherwise).
template <int D>
struct Geo {
  static constexpr int W = D + kRope;
  static constexpr int NK = W / 32;                 // k-steps over the stored channels
  static constexpr int KS = kvk::mla_ksplit(W);     // channel parts per token tile
  static constexpr int NKW = NK / KS;               // k-steps per wave
  static constexpr int TT = 16 * kWaves / KS;       // tokens per iteration
  static constexpr int NBI = TT / 32;               // blocks per iteration
  static constexpr int PH = W + 16;                 // tile row pitch (halfs): W/2 + 8 dwords
  static constexpr int NCT = D / 16;                // latent channel tiles of the product
  static constexpr int NCTW = (NCT + kWaves - 1) / kWaves;  // per wave
  static_assert(NK % KS == 0, "channel parts must split the k-steps evenly");
};

constexpr int kMaxTT = 16 * kWaves;                   // tokens per iteration at KS = 1
constexpr int kTileHalfs = kMaxTT * (256 + kRope + 16);  // the largest TT * PH over widths up to 512
constexpr int kWideTileHalfs = Geo<1024>::TT * Geo<1024>::PH;  // kept width 1024
constexpr int kSP = 20;                               // score rows: 16 tokens + pad (floats)
constexpr int kPP = kMaxTT + 8;                       // probability rows: TT + pad (halfs)
// Kept width 1024 holds the absorbed query of the workgroup's (up to) 32 heads in LDS
// (rows of W + 8 halfs: 16 consecutive rows start 16 distinct 4-bank windows apart).
constexpr int kWideQP = Geo<1024>::W + 8;

// Vector-typed so that 16-byte accesses compile to single b128 LDS instructions.
template <int TILE_HALFS, int Q_HALFS>
struct MlaLds {
  half8 tile[TILE_HALFS / 8];   // fp16 latent rows of the iteration (swizzled)
  half8 q[Q_HALFS > 0 ? Q_HALFS / 8 : 1];  // absorbed query [head][channel] (width 1024 only)
  f4 s[kWaves * 32 * kSP / 4];  // per wave: scores (partial over its channels) [head][token]
  half8 p[32 * kPP / 8];        // probabilities [head][k-slot]
  float alpha[32];
  __device__ __forceinline__ _Float16* tile_h() { return reinterpret_cast<_Float16*>(tile); }
  __device__ __forceinline__ _Float16* p_h() { return reinterpret_cast<_Float16*>(p); }
};

// Element (t, c) of the tile: rows of PH halfs (W/2 + 8 dwords, so consecutive rows
// start 8 banks apart); within a row the 16-byte chunks of rows 4..7 of every 8 swap
// in pairs, so that the tile writes of one phase-A step fall in different banks.  A
// transposed read of the product takes 4 consecutive rows x 16 channels per 16 lanes:
// one swap state, 4 distinct 8-bank windows.
template <int PH>
__device__ __forceinline__ int tile_at(int t, int c) {
  return t * PH + ((((c >> 3) ^ ((t >> 2) & 1))) << 3) + (c & 7);
}

typedef short short4v __attribute__((ext_vector_type(4)));

// Transposed LDS read (ds_read_b64_tr_b16).  Per 16 lanes, lane m names 4 halfs
// (8 bytes); lane i receives, in order, half i % 4 of the lanes i / 4, i / 4 + 4,
// i / 4 + 8 and i / 4 + 12.  So when lane m points at 4 consecutive channels
// 4 (m % 4) .. + 3 of row r0 + m / 4, lane i gets channel i of rows r0 .. r0 + 3.
__device__ __forceinline__ short4v ds_read_tr4(const _Float16* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) short4v*)(const_cast<_Float16*>(p)));
}

// Raw bytes of one wave's share of an iteration (16 tokens x its channel part).
template <int D, int BITS, bool KIVI>
struct MlaRaw {
  static constexpr int NKW = Geo<D>::NKW;
  // per k-step: bf16 8 channels (4 words); int8 2 words; int4 1 word; int2 1 word (half used)
  static constexpr int CW = BITS == 16 ? 4 : (BITS == 8 ? 2 : 1);
  static constexpr int MW = BITS == 16 ? 0 : (KIVI ? NKW : 1);  // metadata words
  uint32_t c[NKW][CW];
  uint32_t m[MW > 0 ? MW : 1];
};

// POL: the cache policy of the loads, non-temporal when one workgroup reads the
// stream, cached when the workgroups of several reader layers read it (the later
// readers then find the lines in L2; non-temporal lines are not kept for them).
// Lane (i = lane % 16, g = lane / 16) of wave part kh holds, at its k-step ks, the
// 8 channels 32 (kh NKW + ks) + 8 g .. + 7 of block row t (its tile's row i): the
// MFMA A-operand layout, which the block's lane-ordered slots follow, so every load
// of a k-step reads one contiguous run of the block.
template <int D, int BITS, bool KIVI, int POL>
__device__ __forceinline__ void mla_issue(MlaRaw<D, BITS, KIVI>& r, Rsrc rs, int soff, int t, int g, int kh) {
  constexpr int W = D + kRope, NKW = Geo<D>::NKW;
  const int j0 = kh * NKW;
  const int kq = (t >> 4) * (W / 32) + j0, i = t & 15;  // first k-step of the part in its tile
  if constexpr (BITS == 16) {
    const int v = 16 * (kq * 64 + i + 16 * g);
#pragma unroll
    for (int ks = 0; ks < NKW; ++ks) {
      const u4v x = __builtin_amdgcn_raw_buffer_load_b128(rs, v + 1024 * ks, soff, POL);
      r.c[ks][0] = x[0]; r.c[ks][1] = x[1]; r.c[ks][2] = x[2]; r.c[ks][3] = x[3];
    }
  } else {
    constexpr int cb = 4 * W * BITS;
    if constexpr (BITS == 8) {
      const int v = 8 * (kq * 64 + i + 16 * g);
#pragma unroll
      for (int ks = 0; ks < NKW; ++ks) {
        const u2v x = __builtin_amdgcn_raw_buffer_load_b64(rs, v + 512 * ks, soff, POL);
        r.c[ks][0] = x[0]; r.c[ks][1] = x[1];
      }
    } else if constexpr (BITS == 4) {
      const int v = 4 * (kq * 64 + i + 16 * g);
#pragma unroll
      for (int ks = 0; ks < NKW; ++ks) r.c[ks][0] = __builtin_amdgcn_raw_buffer_load_b32(rs, v + 256 * ks, soff, POL);
    } else {
      const int v = 4 * ((kq * 16 + i) * 2 + (g >> 1));
#pragma unroll
      for (int ks = 0; ks < NKW; ++ks) r.c[ks][0] = __builtin_amdgcn_raw_buffer_load_b32(rs, v + 128 * ks, soff, POL);
    }
    if constexpr (KIVI) {
      const int v = cb + 4 * (kq * 16 + i);
#pragma unroll
      for (int ks = 0; ks < NKW; ++ks) r.m[ks] = __builtin_amdgcn_raw_buffer_load_b32(rs, v + 64 * ks, soff, POL);
    } else {
      r.m[0] = __builtin_amdgcn_raw_buffer_load_b32(rs, cb + 4 * t, soff, POL);
    }
  }
}

// The 8 fp16 values of k-step ks (see mla_issue).
template <int D, int BITS, bool KIVI>
__device__ __forceinline__ half8 mla_values(const MlaRaw<D, BITS, KIVI>& r, int ks, int g, int kh) {
  if constexpr (BITS == 16) {
    u4v o;
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = bitcast<uint32_t>(bf16x2_to_half2(r.c[ks][e]));
    return bitcast<half8>(o);
  } else {
    constexpr float off = KIVI ? 0.0f : (float)(1 << (BITS - 1));
    half8 u;
    if constexpr (BITS == 8) {
      u = unpack8(r.c[ks][0], r.c[ks][1], off);
    } else if constexpr (BITS == 4) {
      u = unpack4(r.c[ks][0], off);
    } else {
      u = unpack2_half(r.c[ks][0] >> (8 * (g & 1)), off);
    }
    half2v s2, z2;
    if constexpr (KIVI) {
      const uint32_t mm = r.m[ks];
      s2 = bitcast<half2v>(__builtin_amdgcn_perm(mm, mm, 0x01000100u));  // (scale, scale)
      z2 = bitcast<half2v>(__builtin_amdgcn_perm(mm, mm, 0x03020302u));  // (zero, zero)
    } else {
      constexpr int W = D + kRope;
      const int c0 = 32 * (kh * Geo<D>::NKW + ks);  // first channel of the k-step (wave-uniform)
      const uint32_t sb = c0 < D ? (r.m[0] << 16) : (r.m[0] & 0xFFFF0000u);
      s2 = h2s(__uint_as_float(sb));
      z2 = h2s(0.0f);
      (void)W;
    }
    half8 x;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      half2v pr = {u[2 * e], u[2 * e + 1]};
      pr = __builtin_elementwise_fma(pr, s2, z2);
      x[2 * e] = pr[0];
      x[2 * e + 1] = pr[1];
    }
    return x;
  }
}

// Running state of a unit: the product accumulators of the wave's channel tiles
// and, in the softmax threads (8 per head), the head's running max and sum.
template <int D>
struct MlaState {
  f4 o[Geo<D>::NCTW][2];
  float m, l;
};

// The absorbed query fragments of a wave (B operand of the scores: lane (head
// 16 ht + i16, k-group g) holds channels 32 ks + 8 g .. + 7 of its channel part),
// in registers (kept widths up to 512) ...
template <int D>
struct QRegs {
  half8 v[Geo<D>::NKW][2];
  __device__ __forceinline__ half8 get(int ks, int ht) const { return v[ks][ht]; }
};
// ... or read from the LDS copy (kept width 1024).
struct QLds {
  const half8* row[2];  // the lane's first fragment for head tiles 0 and 1
  __device__ __forceinline__ half8 get(int ks, int ht) const { return row[ht][4 * ks]; }
};

// Phase A of an iteration for one wave: values of its 16 tokens x channel part into
// the tile, and its partial scores S^T[token, head] over those channels for the
// chunk's HT head tiles.
template <int D, int BITS, bool KIVI, int HT, class LDS, class Q>
__device__ __forceinline__ void mla_phase_a(const MlaRaw<D, BITS, KIVI>& r, const Q& qreg, LDS& L, int wv, int tt,
                                            int kh, int lane) {
  using G = Geo<D>;
  const int g = lane >> 4, i16 = lane & 15;
  const int row = 16 * tt + i16;
  f4 acc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
#pragma unroll
  for (int ks = 0; ks < G::NKW; ++ks) {
    const half8 x = mla_values<D, BITS, KIVI>(r, ks, g, kh);
    const int c0 = 32 * (kh * G::NKW + ks) + 8 * g;
    L.tile[tile_at<G::PH>(row, c0) >> 3] = x;
    acc[0] = mfma16(x, qreg.get(ks, 0), acc[0]);
    if constexpr (HT == 2) acc[1] = mfma16(x, qreg.get(ks, 1), acc[1]);
  }
#pragma unroll
  for (int ht = 0; ht < HT; ++ht)
    L.s[((wv * 32 + 16 * ht + i16) * kSP + 4 * g) >> 2] = acc[ht];
}

// Phases B (online softmax over the iteration's tokens; the first nvalid count)
// and C (probabilities x latent), after phase A and a barrier, for the chunk's HT
// head tiles (with one tile, the softmax threads of heads 16..31 sit idle: whole
// waves, so the branch is uniform).
template <int D, int HT, class LDS>
__device__ __forceinline__ void mla_phase_bc(MlaState<D>& st, LDS& L, int nvalid, int tid) {
  using G = Geo<D>;
  constexpr int TPB = 2 * kWaves;      // softmax threads per head
  constexpr int TPT = G::TT / TPB;     // tokens per softmax thread
  static_assert(TPT % 4 == 0, "softmax threads read whole f4 score groups");
  const int lane = tid & 63, wv = __builtin_amdgcn_readfirstlane(tid >> 6), g = lane >> 4, i16 = lane & 15;
  static_assert(HT == 2 || 16 * TPB % 64 == 0, "one head tile's softmax threads fill whole waves");
  if (HT == 2 || tid < 16 * TPB) {
    const int h = tid / TPB, p = tid % TPB;
    float x[TPT];
#pragma unroll
    for (int q4 = 0; q4 < TPT / 4; ++q4) {
      const int tok = TPT * p + 4 * q4;  // 4 tokens of one 16-token tile
      const int tt = tok >> 4, r = tok & 15;
      f4 s = L.s[(((tt * G::KS) * 32 + h) * kSP + r) >> 2];
      if constexpr (G::KS == 2) s += L.s[(((tt * 2 + 1) * 32 + h) * kSP + r) >> 2];
#pragma unroll
      for (int e = 0; e < 4; ++e) x[4 * q4 + e] = tok + e < nvalid ? s[e] : -INFINITY;
    }
    float mx = x[0];
#pragma unroll
    for (int e = 1; e < TPT; ++e) mx = fmaxf(mx, x[e]);
    mx = TPB == 8 ? max8(mx) : max16(mx);
    const float mnew = fmaxf(st.m, mx);  // finite: the iteration holds a stored token
    const float alpha = __builtin_amdgcn_exp2f(st.m - mnew);
    float ps = 0.0f;
    _Float16 pv[TPT];  // k-slot j of k-step kk holds token 32 kk + j
#pragma unroll
    for (int e = 0; e < TPT; ++e) {
      pv[e] = (_Float16)__builtin_amdgcn_exp2f(x[e] - mnew);
      ps += (float)pv[e];
    }
    if constexpr (TPT == 8) {
      half8 w8;
#pragma unroll
      for (int e = 0; e < 8; ++e) w8[e] = pv[e];
      L.p[(h * kPP + TPT * p) >> 3] = w8;
    } else {
      short4v w4;
#pragma unroll
      for (int e = 0; e < 4; ++e) w4[e] = bitcast<short>(pv[e]);
      *reinterpret_cast<short4v*>(L.p_h() + h * kPP + TPT * p) = w4;
    }
    st.l = st.l * alpha + (TPB == 8 ? sum8(ps) : sum16(ps));
    st.m = mnew;
    if (p == 0) L.alpha[h] = alpha;
  }
  __syncthreads();
  {
    float al[HT];
    half8 pb[G::TT / 32][HT];  // the probabilities, read once for all channel tiles
#pragma unroll
    for (int ht = 0; ht < HT; ++ht) {
      al[ht] = L.alpha[16 * ht + i16];
#pragma unroll
      for (int kk = 0; kk < G::TT / 32; ++kk) pb[kk][ht] = L.p[((16 * ht + i16) * kPP + 32 * kk + 8 * g) >> 3];
    }
    // Rescale only when some head's running max moved (rare once it has settled).
    bool moved = al[0] != 1.0f;
    if constexpr (HT == 2) moved = moved || al[HT - 1] != 1.0f;
    if (__builtin_amdgcn_ballot_w64(moved)) {
#pragma unroll
      for (int i = 0; i < G::NCTW; ++i)
#pragma unroll
        for (int ht = 0; ht < HT; ++ht) st.o[i][ht] *= al[ht];
    }
    // A operand: lane (channel i16, k-group g) holds tokens 32 kk + 8 g .. + 7.  The
    // swizzle only touches bit 3 of the channel, so tile ct sits 16 kWaves (ct - wv)
    // halfs after tile wv in every row.
    const _Float16* abase[G::TT / 32][2];
#pragma unroll
    for (int kk = 0; kk < G::TT / 32; ++kk) {
      const int r0 = 32 * kk + 8 * g + (i16 >> 2), c = 16 * wv + 4 * (i16 & 3);
      abase[kk][0] = L.tile_h() + tile_at<G::PH>(r0, c);
      abase[kk][1] = L.tile_h() + tile_at<G::PH>(r0 + 4, c);
    }
#pragma unroll
    for (int i = 0; i < G::NCTW; ++i) {
      const int ct = wv + kWaves * i;
      if (G::NCT % kWaves == 0 || ct < G::NCT) {
#pragma unroll
        for (int kk = 0; kk < G::TT / 32; ++kk) {
          const short4v lo = ds_read_tr4(abase[kk][0] + 16 * kWaves * i);
          const short4v hi = ds_read_tr4(abase[kk][1] + 16 * kWaves * i);
          const half8 av = bitcast<half8>(__builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
          for (int ht = 0; ht < HT; ++ht) st.o[i][ht] = mfma16(av, pb[kk][ht], st.o[i][ht]);
        }
      }
    }
  }
}

// sb, units: the split length and the splits of the stream in this call; HT: the
// head tiles of chunk hc (2, or 1 for a last chunk of 16 heads).
template <int D, int BITS, bool KIVI, int POL, int HT, class LDS>
__device__ __forceinline__ void run_mla(const MlaDecodeArgs& a, const MlaItem& it, int rl, int hc,
                                        int b, int u, int sb, int units, LDS& L) {
  using G = Geo<D>;
  constexpr int NR = kvk::mla_ring_depth(G::W, BITS, KIVI ? 1 : 0);
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 4, i16 = lane & 15;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int tt = wv / G::KS, kh = wv % G::KS;
  const int k0 = u * sb;
  const int k1 = min(a.nbf, k0 + sb);
  const int bb = it.block_bytes;
  const uint8_t* stream = a.arena + it.region + (int64_t)b * it.stream_bytes;
  const Rsrc rs = buffer_rsrc(stream, k1 > 0 ? k1 * bb : 0);  // loads past block k1-1 read zeros
  const int trow = 16 * (tt & 1) + i16;                         // token row inside its block
  const int tblk = tt >> 1;                                     // block of the tile in the iteration

  MlaRaw<D, BITS, KIVI> ring[NR];
#pragma unroll
  for (int i = 0; i < NR; ++i) mla_issue<D, BITS, KIVI, POL>(ring[i], rs, (k0 + G::NBI * i + tblk) * bb, trow, g, kh);

  // absorbed query of the chunk's heads over this wave's channel part, fp16
  const _Float16* qsrc = reinterpret_cast<const _Float16*>(a.ws + it.q_off0 + (int64_t)rl * it.q_stride) +
                         ((int64_t)b * a.Hq + 32 * hc) * G::W;
  using QT = typename std::conditional<(D > 512), QLds, QRegs<D>>::type;
  QT qreg;
  if constexpr (D > 512) {
    // the chunk's [16 HT][W] block into LDS; the loop's first barrier orders it before use
    for (int e = tid; e < 16 * HT * (G::W / 8); e += 64 * kWaves) {
      const int h = e / (G::W / 8), c8 = e - h * (G::W / 8);
      L.q[(h * kWideQP >> 3) + c8] = *reinterpret_cast<const half8*>(qsrc + (int64_t)h * G::W + 8 * c8);
    }
#pragma unroll
    for (int ht = 0; ht < 2; ++ht) qreg.row[ht] = L.q + (((16 * ht + i16) * kWideQP + 32 * kh * G::NKW + 8 * g) >> 3);
  } else {
    const _Float16* qb = qsrc + 32 * kh * G::NKW + 8 * g;
#pragma unroll
    for (int ht = 0; ht < HT; ++ht)
#pragma unroll
      for (int ks = 0; ks < G::NKW; ++ks)
        qreg.v[ks][ht] = *reinterpret_cast<const half8*>(qb + (int64_t)(16 * ht + i16) * G::W + 32 * ks);
    // Consume the query here: its first use is then outside the loop, so the loop
    // waits only for the ring entry it uses (a first use inside the loop would make
    // every iteration wait for every load in flight).
#pragma unroll
    for (int ht = 0; ht < HT; ++ht)
#pragma unroll
      for (int ks = 0; ks < G::NKW; ++ks) asm volatile("" ::"v"(qreg.v[ks][ht]));
  }
  MlaState<D> st;
  st.m = -INFINITY;
  st.l = 0.0f;
#pragma unroll
  for (int i = 0; i < G::NCTW; ++i) st.o[i][0] = st.o[i][1] = f4{0.f, 0.f, 0.f, 0.f};

  for (int k = k0; k < k1; k += G::NBI * NR) {
#pragma unroll
    for (int i = 0; i < NR; ++i) {
      const int kb = k + G::NBI * i;                   // first block of the iteration
      const int nvalid = max(0, min(G::TT, 32 * (k1 - kb)));  // uniform
      __syncthreads();                                 // the tile, scores and p are free
      mla_phase_a<D, BITS, KIVI, HT>(ring[i], qreg, L, wv, tt, kh, lane);
      mla_issue<D, BITS, KIVI, POL>(ring[i], rs, (kb + G::NBI * NR + tblk) * bb, trow, g, kh);
      __syncthreads();
      if (nvalid > 0) mla_phase_bc<D, HT>(st, L, nvalid, tid);
    }
  }
  if (u == units - 1 && a.ntail > 0) {  // the bf16 tail block as one more iteration
    MlaRaw<D, 16, false> tr;
    const Rsrc rt = buffer_rsrc(stream + (int64_t)a.nb_cap * bb, tblk == 0 ? 64 * G::W : 0);
    mla_issue<D, 16, false, POL>(tr, rt, 0, trow, g, kh);
    __syncthreads();
    mla_phase_a<D, 16, false, HT>(tr, qreg, L, wv, tt, kh, lane);
    __syncthreads();
    mla_phase_bc<D, HT>(st, L, a.ntail, tid);
  }

  // split partial: m[Hq], l[Hq], o[Hq][D] of this (reader, sequence, split)
  float* rec = reinterpret_cast<float*>(a.ws + it.part_off0 + (int64_t)rl * it.part_stride) +
               ((int64_t)b * it.units_cap + u) * a.Hq * (D + 2);
  if (tid % (2 * kWaves) == 0 && tid / (2 * kWaves) < 16 * HT) {
    const int h = 32 * hc + tid / (2 * kWaves);
    rec[h] = st.m;
    rec[a.Hq + h] = st.l;
  }
  float* orec = rec + 2 * a.Hq;
#pragma unroll
  for (int i = 0; i < G::NCTW; ++i) {
    const int ct = wv + kWaves * i;
    if (ct < G::NCT) {
#pragma unroll
      for (int ht = 0; ht < HT; ++ht) {
        const int h = 32 * hc + 16 * ht + i16;
        *reinterpret_cast<f4*>(orec + (int64_t)h * D + 16 * ct + 4 * g) = st.o[i][ht];
      }
    }
  }
}

// The items of a launch: in the kernel arguments, or (DEV, per-sequence tables) in
// the workspace, read there through the constant address space (nothing writes
// them during the launch), so that the wave-uniform loads go to scalar registers.
// (The host pass of this file parses these functions but never runs them.)
#if defined(__HIP_DEVICE_COMPILE__)
typedef const __attribute__((address_space(4))) MlaItem ConstMlaItem;
#else
typedef const MlaItem ConstMlaItem;
#endif

template <bool DEV>
__device__ __forceinline__ int mla_item_wg_begin(const MlaDecodeArgs& a, int i) {
  if constexpr (DEV) return ((ConstMlaItem*)a.items_dev)[i].wg_begin;
  else return a.items[i].wg_begin;
}

__device__ __forceinline__ MlaItem mla_item_dev(const MlaDecodeArgs& a, int i) {
  return ((ConstMlaItem*)a.items_dev)[i];
}

// A kernel's by-value argument, read in place in the kernel-argument segment (a
// lone struct argument starts at its offset 0) through the constant address space:
// pointers into it that the inlined code selects between then never make the
// compiler copy the 3 KiB struct to private memory first.
template <class T>
__device__ __forceinline__ const T& kernel_args() {
  return *(const T*)__builtin_amdgcn_kernarg_segment_ptr();
}

// The item, reader row, head chunk, sequence, split, split length and splits of
// the stream for workgroup wg; false for the padding workgroups of an item (and for
// splits past the stored blocks of a per-sequence item, whose workgroups are laid
// out for the capacity).  Workgroups of one (sequence, split) for the different
// readers and head chunks sit 8 apart, so that they run on one XCD at about the
// same time and share the stream through its L2.
template <bool DEV>
__device__ __forceinline__ bool mla_locate(const MlaDecodeArgs& a, int wg, int& item, int& rl, int& hc, int& b,
                                           int& u, int& sb, int& units) {
  if (wg >= a.n_wg) return false;
  int lo = 0, hi = a.n_items - 1;  // last item with wg_begin <= wg
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (mla_item_wg_begin<DEV>(a, mid) <= wg) lo = mid;
    else hi = mid - 1;
  }
  const MlaItem& it = DEV ? mla_item_dev(a, lo) : a.items[lo];
  const int R = it.nreaders * it.nhc;
  const int local = wg - it.wg_begin;
  const int grp = local / (8 * R), rem = local - grp * 8 * R;
  const int row = rem >> 3;
  const int unit = 8 * grp + (rem & 7);
  if (unit >= it.nseq * it.units) return false;
  b = unit / it.units;
  u = unit - b * it.units;
  if (it.split_nr > 0) {
    sb = kvk::mla_split_len(it.split_target, it.split_nr, a.nbf);
    units = kvk::mla_units_len(a.nbf, 32 * a.nbf + a.ntail, sb);
  } else {
    sb = it.split_blocks;
    units = it.units;
  }
  if (u >= units) return false;
  item = lo;
  rl = row / it.nhc;
  hc = row - rl * it.nhc;
  return true;
}

// POL: the loads' cache policy for every item of the launch (see mla_issue); the host
// launches single-reader and multi-reader items separately.  Kept widths up to 512:
// two workgroups per CU.
template <bool KIVI, int POL, bool DEV>
__global__ __launch_bounds__(64 * kWaves, 8 / kWaves) void mla_decode_kernel(MlaDecodeArgs) {
  __shared__ MlaLds<kTileHalfs, 0> L;
  const MlaDecodeArgs& a = kernel_args<MlaDecodeArgs>();
  if (!mla_list_ok(a.list_hdr, a.list_hash)) return;  // not this call's list
  int item, rl, hc, b, u, sb, units;
  if (!mla_locate<DEV>(a, blockIdx.x, item, rl, hc, b, u, sb, units)) return;
  const bool two = 32 * hc + 32 <= a.Hq;  // a whole chunk, or the last 16 heads
#define KVK_MLA_CASE(DD, BB)                                                   \
  if (it.d == DD && it.bits == BB) {                                           \
    if (two) run_mla<DD, BB, KIVI, POL, 2>(a, it, rl, hc, b, u, sb, units, L); \
    else run_mla<DD, BB, KIVI, POL, 1>(a, it, rl, hc, b, u, sb, units, L);     \
    return;                                                                    \
  }
#define KVK_MLA_D(DD) KVK_MLA_CASE(DD, 16) KVK_MLA_CASE(DD, 8) KVK_MLA_CASE(DD, 4) KVK_MLA_CASE(DD, 2)
#define KVK_MLA_NARROW \
  KVK_MLA_D(512)       \
  KVK_MLA_D(256)       \
  KVK_MLA_D(128)       \
  KVK_MLA_D(64)        \
  KVK_MLA_D(32)
  if constexpr (DEV) {
    const MlaItem it = mla_item_dev(a, item);
    KVK_MLA_NARROW
  } else {
    const MlaItem& it = a.items[item];
    KVK_MLA_NARROW
  }
#undef KVK_MLA_NARROW
}

// Kept width 1024 (1088 stored channels): the product accumulators take 128
// registers and the iteration's tile 70 KiB of LDS, so one workgroup per CU; the
// absorbed query (136 registers per lane if held there) is read from a 70 KiB LDS
// copy instead.
template <bool KIVI, int POL, bool DEV>
__global__ __launch_bounds__(64 * kWaves, 1) void mla_decode_wide_kernel(MlaDecodeArgs) {
  __shared__ MlaLds<kWideTileHalfs, 32 * kWideQP> L;
  const MlaDecodeArgs& a = kernel_args<MlaDecodeArgs>();
  if (!mla_list_ok(a.list_hdr, a.list_hash)) return;  // not this call's list
  int item, rl, hc, b, u, sb, units;
  if (!mla_locate<DEV>(a, blockIdx.x, item, rl, hc, b, u, sb, units)) return;
  const bool two = 32 * hc + 32 <= a.Hq;
  if constexpr (DEV) {
    const MlaItem it = mla_item_dev(a, item);
    KVK_MLA_D(1024)
  } else {
    const MlaItem& it = a.items[item];
    KVK_MLA_D(1024)
  }
#undef KVK_MLA_D
#undef KVK_MLA_CASE
}

// ---------------------------------------------------------------------------
// C2: merge the splits, then o_h = W_UV[h][:, :d] o_lat
// ---------------------------------------------------------------------------

struct MlaCombineArgs {
  const uint8_t* ws;
  const uint16_t* w_uv;  // [nl][Hq][v][r] bf16
  float* out;            // [nl][B][Hq][v]
  int64_t part_off[KVK_MAX_LAYERS];
  int32_t d_of[KVK_MAX_LAYERS];
  int32_t units[KVK_MAX_LAYERS];
  int32_t units_cap[KVK_MAX_LAYERS];
  const MlaSeqRow* rows;  // per-sequence tables: per (relative layer, sequence) (else NULL)
  const uint64_t* list_hdr;
  uint64_t list_hash;
  int32_t nbf, n_stored;  // per-sequence tables: the splits follow from these
  int32_t B, Hq, Hp, v, r;  // Hp: heads per split partial record (padded)
  int64_t out_lstride;       // elements between consecutive layers' outputs
};

// Sequence b's split partials of relative layer li (fp32 records of Hp (d + 2)), with
// its kept width d, splits U and partial records per sequence UC.
__device__ __forceinline__ const float* combine_src(const MlaCombineArgs& a, int li, int b, int& d, int& U,
                                                    int& UC) {
  if (a.rows) {
    const MlaSeqRow& rw = a.rows[(int64_t)li * a.B + b];
    d = rw.d;
    UC = rw.units_cap;
    U = kvk::mla_units_len(a.nbf, a.n_stored, kvk::mla_split_len(rw.split_target, rw.split_nr, a.nbf));
    return reinterpret_cast<const float*>(a.ws + rw.part_off);
  }
  d = a.d_of[li];
  U = a.units[li];
  UC = a.units_cap[li];
  return reinterpret_cast<const float*>(a.ws + a.part_off[li]) + (int64_t)b * UC * a.Hp * (d + 2);
}

// One workgroup per (layer, head): for 16 sequences at a time, merge the split
// partials by log-sum-exp into o_lat (LDS, bf16 hi + lo), then multiply by
// W_UV[h] on the matrix cores (M = value channels, K = d, N = sequences).  Under
// per-sequence plans K is the widest kept width of the 16, each sequence's o_lat
// zero past its own (the products past it add exact zeros).
template <int DMAX>
__global__ __launch_bounds__(256) void mla_combine_kernel(MlaCombineArgs a) {
  constexpr int PO = DMAX + 8;  // LDS row pitch (bf16)
  constexpr int kMaxU = kvk::kMlaMaxUnits;  // split weights held in LDS per sequence
  __shared__ uint16_t oh[16 * PO], ol[16 * PO];
  __shared__ float wgt[16 * kMaxU];
  const int li = blockIdx.x, h = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, g = lane >> 4, i16 = lane & 15;
  if (!mla_list_ok(a.list_hdr, a.list_hash)) {  // not this call's list: NaN outputs
    for (int e = tid; e < a.B * a.v; e += 256) {
      const int b = e / a.v, j = e - b * a.v;
      a.out[li * a.out_lstride + ((int64_t)b * a.Hq + h) * a.v + j] = __builtin_nanf("");
    }
    return;
  }
  const uint16_t* wv_h = a.w_uv + ((int64_t)li * a.Hq + h) * a.v * a.r;
  for (int b0 = 0; b0 < a.B; b0 += 16) {
    const int nb = min(16, a.B - b0);
    int d = 0;  // the widest kept width of the 16 sequences
    for (int bi = 0; bi < nb; ++bi) {
      int db, U, UC;
      combine_src(a, li, b0 + bi, db, U, UC);
      d = db > d ? db : d;
    }
    __syncthreads();
    // split weights w_u = 2^(m_u - m*) / sum_u 2^(m_u - m*) l_u, one sequence per 16 threads
    {
      const int bi = tid >> 4, p = tid & 15;
      int db = 0, U = 0, UC = 0;
      const float* p0 = bi < nb ? combine_src(a, li, b0 + bi, db, U, UC) : nullptr;
      const int64_t rec = (int64_t)a.Hp * (db + 2);
      float m = -INFINITY;
      if (bi < nb)
        for (int u = p; u < U; u += 16) m = fmaxf(m, p0[u * rec + h]);
      m = max16(m);
      float l = 0.0f;
      if (bi < nb && m > -INFINITY)
        for (int u = p; u < U; u += 16) l += __builtin_amdgcn_exp2f(p0[u * rec + h] - m) * p0[u * rec + a.Hp + h];
      l = sum16(l);
      const float inv = l > 0.0f ? 1.0f / l : 0.0f;
      for (int u = p; u < min(U, kMaxU); u += 16)
        wgt[bi * kMaxU + u] = (bi < nb && inv > 0.0f) ? __builtin_amdgcn_exp2f(p0[u * rec + h] - m) * inv : 0.0f;
    }
    __syncthreads();
    for (int e = tid; e < 4 * d; e += 256) {  // 16 sequences x d channels, 4 channels per step
      const int bi = e / (d / 4), c = 4 * (e - bi * (d / 4));
      f4 x = {0.f, 0.f, 0.f, 0.f};
      if (bi < nb) {
        int db, U, UC;
        const float* p0 = combine_src(a, li, b0 + bi, db, U, UC);
        const int64_t rec = (int64_t)a.Hp * (db + 2);
        if (c < db) {
          const float* o0 = p0 + 2 * a.Hp + (int64_t)h * db + c;
#pragma unroll 4
          for (int u = 0; u < U; ++u) x += wgt[bi * kMaxU + u] * *reinterpret_cast<const f4*>(o0 + u * rec);
        }
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const uint16_t hb = bf16_bits_rne(x[k]);
        oh[bi * PO + c + k] = hb;
        ol[bi * PO + c + k] = bf16_bits_rne(x[k] - bf16_to_f32(hb));
      }
    }
    __syncthreads();
    for (int jt = wv; jt < a.v / 16; jt += 4) {
      // A operands of 16 k-steps of the row tile first (independent loads), then the products
      const uint16_t* wrow = wv_h + (int64_t)(16 * jt + i16) * a.r + 8 * g;
      const int nks = d / 32;
      f4 acc = {0.f, 0.f, 0.f, 0.f};
      for (int k0 = 0; k0 < nks; k0 += 16) {
        u4v wa[16];
#pragma unroll
        for (int ks = 0; ks < 16; ++ks)
          if (k0 + ks < nks) wa[ks] = *reinterpret_cast<const u4v*>(wrow + 32 * (k0 + ks));
#pragma unroll
        for (int ks = 0; ks < 16; ++ks) {
          if (k0 + ks < nks) {
            const int c = 32 * (k0 + ks) + 8 * g;
            const bf16x8 bh = bitcast<bf16x8>(*reinterpret_cast<const u4v*>(&oh[i16 * PO + c]));
            const bf16x8 bl = bitcast<bf16x8>(*reinterpret_cast<const u4v*>(&ol[i16 * PO + c]));
            acc = mfmab(bitcast<bf16x8>(wa[ks]), bh, acc);
            acc = mfmab(bitcast<bf16x8>(wa[ks]), bl, acc);
          }
        }
      }
      if (i16 < nb)  // D[value channel 16 jt + 4g + e][sequence b0 + i16]
        *reinterpret_cast<f4*>(a.out + li * a.out_lstride + ((int64_t)(b0 + i16) * a.Hq + h) * a.v + 16 * jt + 4 * g) = acc;
    }
  }
}

// W_UK from the model's layout ([nl][Hq][nope][r]) to the latent-major one the
// absorption reads ([nl][Hq][r][nope]): one 32 x 32 tile per workgroup through LDS
// (rows of 33 halfs), 8-byte accesses coalesced on both sides.
__global__ __launch_bounds__(256) void mla_arrange_w_uk_kernel(const uint16_t* in, uint16_t* out, int nope, int r) {
  __shared__ uint16_t tile[32][33];
  const int c0 = 32 * blockIdx.x, i0 = 32 * blockIdx.y;  // latent column, nope row of the tile
  const int64_t m = blockIdx.z;                          // (layer, head)
  const uint16_t* src = in + m * nope * r;
  uint16_t* dst = out + m * r * nope;
  const int tid = threadIdx.x, row = tid >> 3, col = 4 * (tid & 7);
  const u2v v = *reinterpret_cast<const u2v*>(src + (int64_t)(i0 + row) * r + c0 + col);
  tile[row][col] = (uint16_t)(v[0] & 0xFFFFu);
  tile[row][col + 1] = (uint16_t)(v[0] >> 16);
  tile[row][col + 2] = (uint16_t)(v[1] & 0xFFFFu);
  tile[row][col + 3] = (uint16_t)(v[1] >> 16);
  __syncthreads();
  u2v w;
  w[0] = (uint32_t)tile[col][row] | ((uint32_t)tile[col + 1][row] << 16);
  w[1] = (uint32_t)tile[col + 2][row] | ((uint32_t)tile[col + 3][row] << 16);
  *reinterpret_cast<u2v*>(dst + (int64_t)(c0 + row) * nope + i0 + col) = w;
}

}  // namespace

namespace kvk {

static kvk_status launch_w2(const MlaCompressArgs& a, int32_t rows, hipStream_t stream);

kvk_status mla_compress_layer(const kvk_table* t, int32_t layer, const void* latent, const void* rope,
                              int32_t in_dtype, int32_t n_tokens, const int32_t* keep_idx, void* arena,
                              hipStream_t stream) {
  const kvk_dims& d = t->d;
  MlaCompressArgs a;
  a.latent = latent;
  a.rope = rope;
  a.keep = keep_idx;
  a.region = static_cast<uint8_t*>(arena) + t->info.layer_offset[layer];
  a.stream_bytes = t->info.stream_bytes[layer];
  a.block_bytes = t->block_bytes[layer];
  a.in_f32 = in_dtype == KVK_F32;
  a.n_tokens = n_tokens;
  a.n_stored = d.keep_tokens > 0 ? d.keep_tokens : n_tokens;
  a.nbf = a.n_stored / KVK_GROUP;
  a.nb_cap = t->nb_cap;
  a.r = d.latent_dim;
  a.d = t->rank[layer];
  a.bits = t->bits[layer];
  a.kivi = d.qscheme == KVK_Q_KIVI32;
  a.n_seq = 0;
  return launch_w2(a, d.batch, stream);
}

// One W2 launch: blocks x `rows` (sequences of one table, or the batch rows of a.seq_of).
static kvk_status launch_w2(const MlaCompressArgs& a, int32_t rows, hipStream_t stream) {
  const dim3 g3((unsigned)(a.nbf + 1), (unsigned)rows), b3(256);
  if (a.bits == 16) hipLaunchKernelGGL((mla_compress_kernel<16, true>), g3, b3, 0, stream, a);
  else if (a.kivi && a.bits == 8) hipLaunchKernelGGL((mla_compress_kernel<8, true>), g3, b3, 0, stream, a);
  else if (a.kivi && a.bits == 4) hipLaunchKernelGGL((mla_compress_kernel<4, true>), g3, b3, 0, stream, a);
  else if (a.kivi) hipLaunchKernelGGL((mla_compress_kernel<2, true>), g3, b3, 0, stream, a);
  else if (a.bits == 8) hipLaunchKernelGGL((mla_compress_kernel<8, false>), g3, b3, 0, stream, a);
  else if (a.bits == 4) hipLaunchKernelGGL((mla_compress_kernel<4, false>), g3, b3, 0, stream, a);
  else hipLaunchKernelGGL((mla_compress_kernel<2, false>), g3, b3, 0, stream, a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(KVK_ERR_DEVICE, "MLA compress launch: %s", hipGetErrorString(e));
  return KVK_OK;
}

kvk_status mla_compress_layer_batched(const kvk_table* t, int32_t layer, const void* latent, const void* rope,
                                      int32_t in_dtype, int32_t n_tokens, const int32_t* keep_idx, void* arena,
                                      hipStream_t stream) {
  const kvk_dims& d = t->d;
  // One launch per (kept width, bit-width) for the sequences whose plans store the
  // layer so; each sequence is written exactly as its one-sequence table writes it.
  std::vector<char> done(d.batch, 0);
  for (int b0 = 0; b0 < d.batch; ++b0) {
    const kvk_table* s0 = t->seq[b0];
    if (done[b0] || s0->plan[layer].inherit) continue;
    MlaCompressArgs a;
    a.latent = latent;
    a.rope = rope;
    a.keep = keep_idx;
    a.region = static_cast<uint8_t*>(arena);
    a.stream_bytes = s0->info.stream_bytes[layer];
    a.block_bytes = s0->block_bytes[layer];
    a.in_f32 = in_dtype == KVK_F32;
    a.n_tokens = n_tokens;
    a.n_stored = d.keep_tokens > 0 ? d.keep_tokens : n_tokens;
    a.nbf = a.n_stored / KVK_GROUP;
    a.nb_cap = t->nb_cap;
    a.r = d.latent_dim;
    a.d = s0->rank[layer];
    a.bits = s0->bits[layer];
    a.kivi = d.qscheme == KVK_Q_KIVI32;
    a.n_seq = 0;
    for (int b = b0; b < d.batch; ++b) {
      const kvk_table* s = t->seq[b];
      if (done[b] || s->plan[layer].inherit || s->rank[layer] != a.d || s->bits[layer] != a.bits) continue;
      done[b] = 1;
      a.seq_of[a.n_seq] = b;
      a.seq_region[a.n_seq] = t->seq_base[b] + s->info.layer_offset[layer];
      if (++a.n_seq == kMlaWriteSeqs) {
        const kvk_status st = launch_w2(a, a.n_seq, stream);
        if (st != KVK_OK) return st;
        a.n_seq = 0;
      }
    }
    if (a.n_seq > 0) {
      const kvk_status st = launch_w2(a, a.n_seq, stream);
      if (st != KVK_OK) return st;
    }
  }
  return KVK_OK;
}

kvk_status mla_append_token(const kvk_table* t, int32_t l0, int32_t l1, const void* latent, const void* rope,
                            int32_t in_dtype, int32_t n_stored, void* arena, hipStream_t stream) {
  const kvk_dims& d = t->d;
  MlaAppendArgs a;
  a.latent = latent;
  a.rope = rope;
  a.arena = static_cast<uint8_t*>(arena);
  a.in_f32 = in_dtype == KVK_F32;
  a.pos = n_stored;
  a.nb_cap = t->nb_cap;
  a.B = d.batch;
  a.r = d.latent_dim;
  // one item per anchor (over all sequences), or per (sequence, anchor of its plan)
  const bool per_seq = !t->seq.empty();
  std::vector<MlaAppendItem> items;
  for (int b = 0; b < (per_seq ? d.batch : 1); ++b) {
    const kvk_table* st = per_seq ? t->seq[b] : t;
    for (int l = l0; l < l1; ++l) {
      if (st->plan[l].inherit) continue;  // an inheriting layer stores nothing (§2.1)
      MlaAppendItem it;
      it.region = (per_seq ? t->seq_base[b] : 0) + st->info.layer_offset[l];
      it.stream_bytes = (int32_t)st->info.stream_bytes[l];
      it.block_bytes = (int32_t)st->block_bytes[l];
      it.bits = st->bits[l];
      it.row = l - l0;
      it.d = st->rank[l];
      it.seq = per_seq ? b : -1;
      items.push_back(it);
    }
  }
  const dim3 b3(256);
  for (size_t i0 = 0; i0 < items.size(); i0 += KVK_MAX_LAYERS) {
    const int n = (int)std::min<size_t>(KVK_MAX_LAYERS, items.size() - i0);
    std::copy(items.begin() + i0, items.begin() + i0 + n, a.items);
    const dim3 g3(per_seq ? 1u : (unsigned)d.batch, (unsigned)n);
    if (d.qscheme == KVK_Q_KIVI32) hipLaunchKernelGGL(mla_append_kernel<true>, g3, b3, 0, stream, a);
    else hipLaunchKernelGGL(mla_append_kernel<false>, g3, b3, 0, stream, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(KVK_ERR_DEVICE, "MLA append launch: %s", hipGetErrorString(e));
  }
  return KVK_OK;
}

static kvk_status launch_w2p(const MlaProjectArgs& a, int bits, bool kivi, int32_t rows, hipStream_t stream);

kvk_status mla_compress_layer_project(const kvk_table* t, int32_t layer, const void* x, const void* w_dkv,
                                      int32_t d_model, const void* rope, int32_t n_tokens,
                                      const int32_t* keep_idx, void* arena, void* latent_out, hipStream_t stream) {
  const kvk_dims& d = t->d;
  MlaProjectArgs a;
  a.x = static_cast<const uint16_t*>(x);
  a.w = static_cast<const uint16_t*>(w_dkv);
  a.rope = static_cast<const uint16_t*>(rope);
  a.keep = keep_idx;
  a.region = static_cast<uint8_t*>(arena) + t->info.layer_offset[layer];
  a.latent_out = static_cast<uint16_t*>(latent_out);
  a.stream_bytes = t->info.stream_bytes[layer];
  a.block_bytes = t->block_bytes[layer];
  a.n_tokens = n_tokens;
  a.n_stored = d.keep_tokens > 0 ? d.keep_tokens : n_tokens;
  a.nbf = a.n_stored / KVK_GROUP;
  a.nb_cap = t->nb_cap;
  a.H = d_model;
  a.d = t->rank[layer];
  a.n_seq = 0;
  return launch_w2p(a, t->bits[layer], d.qscheme == KVK_Q_KIVI32, d.batch, stream);
}

kvk_status mla_compress_layer_project_batched(const kvk_table* t, int32_t layer, const void* x, const void* w_dkv,
                                              int32_t d_model, const void* rope, int32_t n_tokens,
                                              const int32_t* keep_idx, void* arena, hipStream_t stream) {
  const kvk_dims& d = t->d;
  // One launch per (kept width, bit-width) for the sequences whose plans store the
  // layer so; each sequence is written exactly as its one-sequence table writes it.
  std::vector<char> done(d.batch, 0);
  for (int b0 = 0; b0 < d.batch; ++b0) {
    const kvk_table* s0 = t->seq[b0];
    if (done[b0] || s0->plan[layer].inherit) continue;
    MlaProjectArgs a;
    a.x = static_cast<const uint16_t*>(x);
    a.w = static_cast<const uint16_t*>(w_dkv);
    a.rope = static_cast<const uint16_t*>(rope);
    a.keep = keep_idx;
    a.region = static_cast<uint8_t*>(arena);
    a.latent_out = nullptr;
    a.stream_bytes = s0->info.stream_bytes[layer];
    a.block_bytes = s0->block_bytes[layer];
    a.n_tokens = n_tokens;
    a.n_stored = d.keep_tokens > 0 ? d.keep_tokens : n_tokens;
    a.nbf = a.n_stored / KVK_GROUP;
    a.nb_cap = t->nb_cap;
    a.H = d_model;
    a.d = s0->rank[layer];
    a.n_seq = 0;
    const int bits = s0->bits[layer];
    for (int b = b0; b < d.batch; ++b) {
      const kvk_table* s = t->seq[b];
      if (done[b] || s->plan[layer].inherit || s->rank[layer] != a.d || s->bits[layer] != bits) continue;
      done[b] = 1;
      a.seq_of[a.n_seq] = b;
      a.seq_region[a.n_seq] = t->seq_base[b] + s->info.layer_offset[layer];
      if (++a.n_seq == kMlaWriteSeqs) {
        const kvk_status st = launch_w2p(a, bits, d.qscheme == KVK_Q_KIVI32, a.n_seq, stream);
        if (st != KVK_OK) return st;
        a.n_seq = 0;
      }
    }
    if (a.n_seq > 0) {
      const kvk_status st = launch_w2p(a, bits, d.qscheme == KVK_Q_KIVI32, a.n_seq, stream);
      if (st != KVK_OK) return st;
    }
  }
  return KVK_OK;
}

// One projected-write launch: `rows` sequences (of one table, or the batch rows of
// a.seq_of) at the arguments' kept width and the given bit-width.
static kvk_status launch_w2p(const MlaProjectArgs& a, int bits, bool kivi, int32_t rows, hipStream_t stream) {
  const int tok = a.d > 512 ? ProjGeo<1024>::TOK : ProjGeo<512>::TOK;  // stored tokens per workgroup
  const dim3 g3((unsigned)((a.nbf + 1 + tok / 32 - 1) / (tok / 32)), (unsigned)rows), b3(512);
#define KVK_PROJ(DD)                                                                                          \
  if (a.d == DD) {                                                                                            \
    if (bits == 16) hipLaunchKernelGGL((mla_project_kernel<DD, 16, true>), g3, b3, 0, stream, a);              \
    else if (kivi && bits == 8) hipLaunchKernelGGL((mla_project_kernel<DD, 8, true>), g3, b3, 0, stream, a);  \
    else if (kivi && bits == 4) hipLaunchKernelGGL((mla_project_kernel<DD, 4, true>), g3, b3, 0, stream, a);  \
    else if (kivi) hipLaunchKernelGGL((mla_project_kernel<DD, 2, true>), g3, b3, 0, stream, a);               \
    else if (bits == 8) hipLaunchKernelGGL((mla_project_kernel<DD, 8, false>), g3, b3, 0, stream, a);         \
    else if (bits == 4) hipLaunchKernelGGL((mla_project_kernel<DD, 4, false>), g3, b3, 0, stream, a);         \
    else hipLaunchKernelGGL((mla_project_kernel<DD, 2, false>), g3, b3, 0, stream, a);                        \
  }
  KVK_PROJ(1024) else KVK_PROJ(512) else KVK_PROJ(256) else KVK_PROJ(128) else KVK_PROJ(64) else KVK_PROJ(32)
  else return fail(KVK_ERR_UNSUPPORTED, "projected write: kept width %d", a.d);
#undef KVK_PROJ
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(KVK_ERR_DEVICE, "MLA projected write launch: %s", hipGetErrorString(e));
  return KVK_OK;
}

kvk_status mla_debug_dequantize(const kvk_table* t, int32_t layer, int32_t n_stored, const void* arena,
                                float* c_out, float* r_out, hipStream_t stream) {
  const kvk_dims& d = t->d;
  const int a = t->info.anchor_of[layer];
  const int W = t->rank[a] + d.rope_dim;
  const int64_t total = (int64_t)d.batch * n_stored * W;
  const int64_t grid = (total + 255) / 256;
  if (grid > 0x7fffffffLL) return fail(KVK_ERR_UNSUPPORTED, "grid too large");
  hipLaunchKernelGGL(mla_dequant_kernel, dim3((unsigned)grid), dim3(256), 0, stream,
                     static_cast<const uint8_t*>(arena) + t->info.layer_offset[a], t->info.stream_bytes[a],
                     t->block_bytes[a], t->nb_cap, n_stored, d.batch, t->rank[a], t->bits[a],
                     d.qscheme == KVK_Q_KIVI32 ? 1 : 0, c_out, r_out);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(KVK_ERR_DEVICE, "MLA dequantise launch: %s", hipGetErrorString(e));
  return KVK_OK;
}

// D2 launch class k: bit 0 the cached load policy (items whose stream several
// workgroups read), bit 1 the width-1024 kernel; a.n_wg workgroups.
kvk_status launch_mla_d2(const MlaDecodeArgs& a, int k, bool kivi, hipStream_t stream) {
  const dim3 grid((unsigned)a.n_wg), blk(64 * kWaves);
  const bool dev = a.items_dev != nullptr;
#define KVK_D2(KERNEL, KV, PO)                                                                          \
  if (dev) hipLaunchKernelGGL((KERNEL<KV, PO, true>), grid, blk, 0, stream, a);                        \
  else hipLaunchKernelGGL((KERNEL<KV, PO, false>), grid, blk, 0, stream, a);
  switch (k + 4 * (kivi ? 1 : 0)) {
    case 0: KVK_D2(mla_decode_kernel, false, kStreamPolicy) break;
    case 1: KVK_D2(mla_decode_kernel, false, 0) break;
    case 2: KVK_D2(mla_decode_wide_kernel, false, kStreamPolicy) break;
    case 3: KVK_D2(mla_decode_wide_kernel, false, 0) break;
    case 4: KVK_D2(mla_decode_kernel, true, kStreamPolicy) break;
    case 5: KVK_D2(mla_decode_kernel, true, 0) break;
    case 6: KVK_D2(mla_decode_wide_kernel, true, kStreamPolicy) break;
    default: KVK_D2(mla_decode_wide_kernel, true, 0) break;
  }
#undef KVK_D2
  const hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(KVK_ERR_DEVICE, "MLA decode launch: %s", hipGetErrorString(err));
  return KVK_OK;
}

kvk_status mla_decode_splits(const kvk_table* t, int32_t l0, int32_t l1, const void* q, int32_t q_dtype,
                             int32_t n_stored, float scale, const void* w_uk, const void* arena,
                             void* workspace, hipStream_t stream, int64_t q_lstride) {
  const kvk_dims& d = t->d;
  MlaWorkspace ws;
  mla_workspace(t, l0, l1, &ws);
  uint8_t* wsb = static_cast<uint8_t*>(workspace);

  // A1: absorbed queries of every layer of the range
  MlaAbsorbArgs aa;
  aa.q = q;
  aa.w_ukt = static_cast<const uint16_t*>(w_uk);
  aa.ws = wsb;
  aa.q_f32 = q_dtype == KVK_F32;
  aa.B = d.batch;
  aa.Hq = d.n_q_heads;
  aa.Hp = mla_heads_padded(d.n_q_heads);
  aa.q_lstride = q_lstride > 0 ? q_lstride : (int64_t)d.batch * d.n_q_heads * (d.nope_dim + d.rope_dim);
  aa.nope = d.nope_dim;
  aa.r = d.latent_dim;
  aa.scale_log2 = scale * kLog2e;
  for (int l = l0; l < l1; ++l) {
    aa.q_off[l - l0] = ws.q_off[l];
    aa.d_of[l - l0] = t->rank[t->info.anchor_of[l]];
  }
  aa.rows = nullptr;
  aa.list_hdr = nullptr;
  aa.list_hash = 0;
  hipLaunchKernelGGL(mla_absorb_kernel, dim3((unsigned)(l1 - l0), (unsigned)aa.Hp, (unsigned)((d.batch + 15) / 16)),
                     dim3(256), 0, stream, aa);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(KVK_ERR_DEVICE, "MLA absorb launch: %s", hipGetErrorString(e));

  // D2: one item per distinct anchor read by the range (depth sharing, §2.1)
  const int nbf = n_stored / KVK_GROUP, ntail = n_stored % KVK_GROUP;
  if (n_stored == 0) {
    // no tokens: every partial is (m = -inf, l = 0, o = 0); the merge then yields zeros
    // and needs no partials, so nothing is launched here.
    return KVK_OK;
  }
  // Up to four launches: items whose stream one workgroup reads (non-temporal loads)
  // and items read by the workgroups of several reader layers or head chunks
  // (cached), each for kept widths up to 512 and for 1024 (its own kernel).
  // Launch k + 2 w: policy k, width class w.
  MlaDecodeArgs args[4];
  int64_t wgs_of[4] = {0, 0, 0, 0};
  for (MlaDecodeArgs& a : args) {
    a.arena = static_cast<const uint8_t*>(arena);
    a.ws = wsb;
    a.items_dev = nullptr;
    a.list_hdr = nullptr;
    a.list_hash = 0;
    a.B = d.batch;
    a.Hq = mla_heads_padded(d.n_q_heads);
    a.nbf = nbf;
    a.ntail = ntail;
    a.nb_cap = t->nb_cap;
    a.n_items = 0;
  }
  auto flush = [&](int k) -> kvk_status {
    MlaDecodeArgs& a = args[k];
    int64_t& wgs = wgs_of[k];
    if (a.n_items == 0) return KVK_OK;
    // Launch order: the widest kept width first (then the most bits), as the
    // per-sequence lists order their items.  Measured on the 32-layer latent stack
    // (A1 + D2): int4 648 / 605 -> 587 / 568 us, bf16 916 / 884 -> 883 us against
    // layer order; the narrowest first gave about the same.
    std::stable_sort(a.items, a.items + a.n_items, [](const MlaItem& x, const MlaItem& y) {
      return x.d != y.d ? x.d > y.d : x.bits > y.bits;
    });
    wgs = 0;
    for (int i = 0; i < a.n_items; ++i) {
      MlaItem& it = a.items[i];
      it.wg_begin = (int32_t)wgs;
      wgs += ((int64_t)it.nseq * it.units + 7) / 8 * 8 * it.nreaders * it.nhc;
    }
    if (wgs > 0x7fffffffLL) return fail(KVK_ERR_UNSUPPORTED, "too many MLA decode workgroups");
    a.n_wg = (int32_t)wgs;
    const kvk_status st = launch_mla_d2(a, k, d.qscheme == KVK_Q_KIVI32, stream);
    a.n_items = 0;
    wgs = 0;
    return st;
  };
  const int nhc = mla_head_chunks(d.n_q_heads);
  // A class with more items than one launch's arguments hold runs as launches of
  // equal item counts (a short last launch would run alone, far from filling the GPU).
  int n_class[4] = {0, 0, 0, 0}, per_launch[4];
  for (int l = l0; l < l1;) {
    const int anc = t->info.anchor_of[l];
    const int re = t->next_anchor[anc] < l1 ? t->next_anchor[anc] : l1;
    ++n_class[((re - l) * nhc > 1 ? 1 : 0) + (t->rank[anc] > 512 ? 2 : 0)];
    l = re;
  }
  for (int k = 0; k < 4; ++k) {
    const int nl = (n_class[k] + kMaxItems - 1) / kMaxItems;
    per_launch[k] = nl > 0 ? (n_class[k] + nl - 1) / nl : kMaxItems;
  }
  for (int l = l0; l < l1;) {
    const int anc = t->info.anchor_of[l];
    const int re = t->next_anchor[anc] < l1 ? t->next_anchor[anc] : l1;  // readers [l, re)
    const int k = ((re - l) * nhc > 1 ? 1 : 0) + (t->rank[anc] > 512 ? 2 : 0);
    MlaDecodeArgs& a = args[k];
    int64_t& wgs = wgs_of[k];
    if (a.n_items == per_launch[k]) {
      const kvk_status st = flush(k);
      if (st != KVK_OK) return st;
    }
    MlaItem& it = a.items[a.n_items++];
    it.region = t->info.layer_offset[anc];
    it.q_off0 = ws.q_off[l];
    it.q_stride = re - l > 1 ? ws.q_off[l + 1] - ws.q_off[l] : 0;
    it.part_off0 = ws.part_off[l];
    it.part_stride = re - l > 1 ? ws.part_off[l + 1] - ws.part_off[l] : 0;
    it.stream_bytes = (int32_t)t->info.stream_bytes[anc];
    it.block_bytes = (int32_t)t->block_bytes[anc];
    it.d = t->rank[anc];
    it.bits = t->bits[anc];
    it.nreaders = re - l;
    it.nhc = nhc;
    it.split_blocks = mla_split_blocks_for(t, anc, nbf);
    it.units = mla_units(t, anc, n_stored);
    it.units_cap = ws.units_cap[l];
    it.wg_begin = (int32_t)wgs;
    it.nseq = d.batch;
    it.split_target = 0;
    it.split_nr = 0;
    it.reserved = 0;
    const int64_t units = (int64_t)d.batch * it.units;
    wgs += (units + 7) / 8 * 8 * it.nreaders * nhc;
    l = re;
  }
  for (int k = 0; k < 4; ++k) {
    const kvk_status st = flush(k);
    if (st != KVK_OK) return st;
  }
  return KVK_OK;
}

kvk_status mla_absorb_rows(const kvk_table* t, const void* q, int32_t rows, const void* w_uk, void* out,
                           float scale, hipStream_t stream) {
  const kvk_dims& d = t->d;
  MlaAbsorbArgs aa;
  aa.q = q;
  aa.w_ukt = static_cast<const uint16_t*>(w_uk);
  aa.ws = static_cast<uint8_t*>(out);
  aa.q_f32 = 0;
  aa.B = rows;
  aa.Hq = d.n_q_heads;
  aa.Hp = mla_heads_padded(d.n_q_heads);
  aa.nope = d.nope_dim;
  aa.r = d.latent_dim;
  aa.q_lstride = (int64_t)rows * d.n_q_heads * (d.nope_dim + d.rope_dim);
  aa.scale_log2 = scale * kLog2e;
  aa.q_off[0] = 0;
  aa.d_of[0] = d.latent_dim;  // the full width
  aa.rows = nullptr;
  aa.list_hdr = nullptr;
  aa.list_hash = 0;
  hipLaunchKernelGGL(mla_absorb_kernel, dim3(1u, (unsigned)aa.Hp, (unsigned)((rows + 15) / 16)), dim3(256), 0, stream, aa);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(KVK_ERR_DEVICE, "MLA absorb launch: %s", hipGetErrorString(e));
  return KVK_OK;
}

kvk_status mla_decode_merge(const kvk_table* t, int32_t l0, int32_t l1, int32_t n_stored, const void* w_uv,
                            const void* workspace, float* out, hipStream_t stream, int64_t out_lstride) {
  const kvk_dims& d = t->d;
  MlaWorkspace ws;
  mla_workspace(t, l0, l1, &ws);
  MlaCombineArgs c;
  c.ws = static_cast<const uint8_t*>(workspace);
  c.w_uv = static_cast<const uint16_t*>(w_uv);
  c.out = out;
  c.B = d.batch;
  c.Hq = d.n_q_heads;
  c.Hp = mla_heads_padded(d.n_q_heads);
  c.out_lstride = out_lstride > 0 ? out_lstride : (int64_t)d.batch * d.n_q_heads * d.v_dim;
  c.v = d.v_dim;
  c.r = d.latent_dim;
  c.rows = nullptr;
  c.list_hdr = nullptr;
  c.list_hash = 0;
  c.nbf = 0;
  c.n_stored = 0;
  int dmax = 0;
  for (int l = l0; l < l1; ++l) {
    const int anc = t->info.anchor_of[l];
    c.part_off[l - l0] = ws.part_off[l];
    c.d_of[l - l0] = t->rank[anc];
    c.units[l - l0] = n_stored > 0 ? mla_units(t, anc, n_stored) : 0;  // none: o = 0
    c.units_cap[l - l0] = ws.units_cap[l];
    dmax = t->rank[anc] > dmax ? t->rank[anc] : dmax;
  }
  const dim3 grid((unsigned)(l1 - l0), (unsigned)d.n_q_heads);
  if (dmax > 512) hipLaunchKernelGGL(mla_combine_kernel<1024>, grid, dim3(256), 0, stream, c);
  else hipLaunchKernelGGL(mla_combine_kernel<512>, grid, dim3(256), 0, stream, c);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(KVK_ERR_DEVICE, "MLA combine launch: %s", hipGetErrorString(e));
  return KVK_OK;
}

// ---------------------------------------------------------------------------
// Per-sequence plans (§2.3, eq. (3) with the rank axis): one launch per phase for the
// whole batch.  The work list (a row per (layer, sequence), an item per (sequence,
// anchor) in each D2 launch class) is written once per workspace and layer range by
// kvk_decode_setup; every decode call rebuilds it on the host only to check that the
// workspace holds it (its hash) and to size the launches.  The splits follow from
// the stored length in the kernels (each row and item carries its anchor's split
// rule), so the list does not depend on it.  Sequence b's absorbed queries and
// partials sit in its own part of the workspace, laid out as its one-sequence table
// lays them out, the parts one after the other after the list.
// ---------------------------------------------------------------------------

MlaSeqList::MlaSeqList() = default;
MlaSeqList::~MlaSeqList() = default;

kvk_status mla_seq_list(const kvk_table* t, int32_t l0, int32_t l1, MlaSeqList& L, bool image) {
  const kvk_dims& d = t->d;
  const int32_t nl = l1 - l0, B = d.batch;
  const int nhc = mla_head_chunks(d.n_q_heads);
  // items per launch class
  int32_t n_k[4] = {0, 0, 0, 0};
  for (int b = 0; b < B; ++b) {
    const kvk_table* s = t->seq[b];
    for (int l = l0; l < l1;) {
      const int anc = s->info.anchor_of[l];
      const int re = s->next_anchor[anc] < l1 ? s->next_anchor[anc] : l1;
      ++n_k[((re - l) * nhc > 1 ? 1 : 0) + (s->rank[anc] > 512 ? 2 : 0)];
      l = re;
    }
  }
  int64_t off = 256;
  L.rows_off = off;
  off += round256((int64_t)nl * B * (int64_t)sizeof(MlaSeqRow));
  for (int k = 0; k < 4; ++k) {
    L.items_off[k] = off;
    L.n_items[k] = n_k[k];
    L.n_wg[k] = 0;
    off += round256((int64_t)n_k[k] * (int64_t)sizeof(MlaItem));
  }
  L.bytes = off;
  L.dmax = 0;
  if (!image) return KVK_OK;
  L.img.assign((size_t)L.bytes, 0);
  MlaSeqRow* rows = reinterpret_cast<MlaSeqRow*>(L.img.data() + L.rows_off);
  std::vector<MlaItem> items[4];
  int64_t base = L.bytes;  // sequence b's part of the workspace
  for (int b = 0; b < B; ++b) {
    const kvk_table* s = t->seq[b];
    MlaWorkspace w;
    mla_workspace(s, l0, l1, &w);
    for (int l = l0; l < l1; ++l) {
      const int anc = s->info.anchor_of[l];
      MlaSeqRow& r = rows[(int64_t)(l - l0) * B + b];
      r.q_off = base + w.q_off[l];
      r.part_off = base + w.part_off[l];
      r.d = s->rank[anc];
      r.units_cap = w.units_cap[l];
      mla_split_rule(s, anc, &r.split_target, &r.split_nr);
      L.dmax = r.d > L.dmax ? r.d : L.dmax;
    }
    for (int l = l0; l < l1;) {
      const int anc = s->info.anchor_of[l];
      const int re = s->next_anchor[anc] < l1 ? s->next_anchor[anc] : l1;  // readers [l, re)
      const int k = ((re - l) * nhc > 1 ? 1 : 0) + (s->rank[anc] > 512 ? 2 : 0);
      MlaItem it;
      std::memset(&it, 0, sizeof(it));  // the list is hashed byte for byte: padding too
      it.region = t->seq_base[b] + s->info.layer_offset[anc];
      it.q_off0 = base + w.q_off[l];
      it.q_stride = re - l > 1 ? w.q_off[l + 1] - w.q_off[l] : 0;
      it.part_off0 = base + w.part_off[l];
      it.part_stride = re - l > 1 ? w.part_off[l + 1] - w.part_off[l] : 0;
      it.stream_bytes = (int32_t)s->info.stream_bytes[anc];
      it.block_bytes = (int32_t)s->block_bytes[anc];
      it.d = s->rank[anc];
      it.bits = s->bits[anc];
      it.nreaders = re - l;
      it.nhc = nhc;
      it.units = w.units_cap[l];  // workgroups laid out for the capacity
      it.units_cap = w.units_cap[l];
      it.split_blocks = 0;
      it.wg_begin = 0;
      it.nseq = 1;
      mla_split_rule(s, anc, &it.split_target, &it.split_nr);
      items[k].push_back(it);
      l = re;
    }
    base += w.total;
  }
  // Launch order: the items of one (kept width, bit-width) together, so that the
  // workgroups sharing a CU mostly run the same specialisation of the kernel (each is
  // large; a CU that alternates between them keeps reloading instructions).
  // Workgroup ids go round the 8 XCDs.  An item one workgroup row reads takes its
  // units' workgroups back to back.  An item several rows (readers, head chunks) read
  // keeps the 8-unit groups whose rows sit 8 apart (one XCD per unit); a
  // one-sequence item has fewer than 8 units, so its first workgroup is moved on (by
  // workgroups that exit at once) to the XCD after the previous item's last unit,
  // instead of every such item starting on the same XCD.
  for (int k = 0; k < 4; ++k) {
    std::stable_sort(items[k].begin(), items[k].end(), [](const MlaItem& x, const MlaItem& y) {
      return x.d != y.d ? x.d > y.d : x.bits > y.bits;
    });
    MlaItem* dst = reinterpret_cast<MlaItem*>(L.img.data() + L.items_off[k]);
    int64_t placed = 0;  // units placed so far
    for (size_t i = 0; i < items[k].size(); ++i) {
      MlaItem& it = items[k][i];
      const int64_t R = (int64_t)it.nreaders * nhc;
      if (R == 1) {
        it.wg_begin = (int32_t)L.n_wg[k];
        L.n_wg[k] += it.units;
      } else {
        L.n_wg[k] += ((placed - L.n_wg[k]) % 8 + 8) % 8;
        it.wg_begin = (int32_t)L.n_wg[k];
        L.n_wg[k] += (int64_t)(it.units + 7) / 8 * 8 * R;
      }
      placed += it.units;
      std::memcpy(dst + i, &it, sizeof(MlaItem));
    }
  }
  for (int k = 0; k < 4; ++k)
    if (L.n_wg[k] > 0x7fffffffLL) return fail(KVK_ERR_UNSUPPORTED, "too many MLA decode workgroups");
  L.hash = fnv1a64(L.img.data() + 256, L.img.size() - 256);
  uint64_t* hdr = reinterpret_cast<uint64_t*>(L.img.data());
  hdr[0] = kMlaListMagic;
  hdr[1] = L.hash;
  return KVK_OK;
}

kvk_status mla_decode_batched(const kvk_table* t, int32_t l0, int32_t l1, const void* q, int32_t q_dtype,
                              int32_t n_stored, float scale, const void* w_uk, const void* w_uv,
                              const void* arena, float* out, void* workspace, hipStream_t stream, bool splits,
                              bool merge) {
  const kvk_dims& d = t->d;
  // The list depends on the table and the layer range only: its set-up recorded
  // where it sits and the launch sizes (the kernels check its hash in the workspace).
  kvk_table::DecodeSetup L;
  {
    bool ready = false;
    std::lock_guard<std::mutex> lock(t->setup_mu);
    for (const kvk_table::DecodeSetup& su : t->setups)
      if (su.workspace == workspace && su.l0 == l0 && su.l1 == l1) {
        L = su;
        ready = true;
      }
    if (!ready)
      return fail(KVK_ERR_INVALID,
                  "per-sequence plans: call kvk_decode_setup for layers [%d, %d) on this workspace first", l0, l1);
  }
  uint8_t* wsb = static_cast<uint8_t*>(workspace);
  const uint64_t* hdr = reinterpret_cast<const uint64_t*>(wsb);
  const int32_t nl = l1 - l0, nbf = n_stored / KVK_GROUP, ntail = n_stored % KVK_GROUP;
  const int32_t Hp = mla_heads_padded(d.n_q_heads);
  const int64_t qw = d.nope_dim + d.rope_dim;
  if (splits) {
    MlaAbsorbArgs aa;
    aa.q = q;
    aa.w_ukt = static_cast<const uint16_t*>(w_uk);
    aa.ws = wsb;
    aa.rows = reinterpret_cast<const MlaSeqRow*>(wsb + L.rows_off);
    aa.list_hdr = hdr;
    aa.list_hash = L.hash;
    aa.q_f32 = q_dtype == KVK_F32;
    aa.B = d.batch;
    aa.Hq = d.n_q_heads;
    aa.Hp = Hp;
    aa.nope = d.nope_dim;
    aa.r = d.latent_dim;
    aa.q_lstride = (int64_t)d.batch * d.n_q_heads * qw;
    aa.scale_log2 = scale * kLog2e;
    hipLaunchKernelGGL(mla_absorb_kernel, dim3((unsigned)nl, (unsigned)Hp, (unsigned)((d.batch + 15) / 16)), dim3(256), 0,
                       stream, aa);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(KVK_ERR_DEVICE, "MLA absorb launch: %s", hipGetErrorString(e));
    if (n_stored > 0) {  // none stored: the merge needs no partials
      for (int k = 0; k < 4; ++k) {
        if (L.n_items[k] == 0) continue;
        MlaDecodeArgs a;
        a.arena = static_cast<const uint8_t*>(arena);
        a.ws = wsb;
        a.items_dev = reinterpret_cast<const MlaItem*>(wsb + L.items_off[k]);
        a.list_hdr = hdr;
        a.list_hash = L.hash;
        a.n_items = L.n_items[k];
        a.n_wg = (int32_t)L.n_wg[k];
        a.B = d.batch;
        a.Hq = Hp;
        a.nbf = nbf;
        a.ntail = ntail;
        a.nb_cap = t->nb_cap;
        if (kvk_status st = launch_mla_d2(a, k, d.qscheme == KVK_Q_KIVI32, stream)) return st;
      }
    }
  }
  if (merge) {
    MlaCombineArgs c;
    c.ws = wsb;
    c.w_uv = static_cast<const uint16_t*>(w_uv);
    c.out = out;
    c.rows = reinterpret_cast<const MlaSeqRow*>(wsb + L.rows_off);
    c.list_hdr = hdr;
    c.list_hash = L.hash;
    c.nbf = nbf;
    c.n_stored = n_stored;
    c.B = d.batch;
    c.Hq = d.n_q_heads;
    c.Hp = Hp;
    c.v = d.v_dim;
    c.r = d.latent_dim;
    c.out_lstride = (int64_t)d.batch * d.n_q_heads * d.v_dim;
    const dim3 grid((unsigned)nl, (unsigned)d.n_q_heads);
    if (L.dmax > 512) hipLaunchKernelGGL(mla_combine_kernel<1024>, grid, dim3(256), 0, stream, c);
    else hipLaunchKernelGGL(mla_combine_kernel<512>, grid, dim3(256), 0, stream, c);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(KVK_ERR_DEVICE, "MLA combine launch: %s", hipGetErrorString(e));
  }
  return KVK_OK;
}

}  // namespace kvk

// Absorption-ready W_UK (App. C.2): the transpose of every (layer, head) matrix.
extern "C" kvk_status kvk_mla_arrange_w_uk(const void* w_uk, int32_t n_layers, int32_t n_heads, int32_t nope_dim,
                                           int32_t latent_dim, void* out, hipStream_t stream) {
  if (!w_uk || !out) return kvk::fail(KVK_ERR_INVALID, "kvk_mla_arrange_w_uk: NULL buffer");
  if (n_layers < 1 || n_layers > KVK_MAX_LAYERS || n_heads < 1 || n_heads > 256)
    return kvk::fail(KVK_ERR_INVALID, "kvk_mla_arrange_w_uk: %d layers x %d heads", n_layers, n_heads);
  if (nope_dim < 32 || nope_dim % 32 || latent_dim < 32 || latent_dim % 32)
    return kvk::fail(KVK_ERR_INVALID, "kvk_mla_arrange_w_uk: nope_dim %d and latent_dim %d must be multiples of 32",
                     nope_dim, latent_dim);
  if ((reinterpret_cast<uintptr_t>(w_uk) & 15) || (reinterpret_cast<uintptr_t>(out) & 15))
    return kvk::fail(KVK_ERR_INVALID, "kvk_mla_arrange_w_uk: misaligned buffer (16 bytes required)");
  if (w_uk == out) return kvk::fail(KVK_ERR_INVALID, "kvk_mla_arrange_w_uk: the output may not alias the input");
  if (kvk_status st = kvk::check_gpu_buffers({w_uk, out}, "kvk_mla_arrange_w_uk")) return st;
  const dim3 grid((unsigned)(latent_dim / 32), (unsigned)(nope_dim / 32), (unsigned)(n_layers * n_heads));
  hipLaunchKernelGGL(mla_arrange_w_uk_kernel, grid, dim3(256), 0, stream, static_cast<const uint16_t*>(w_uk),
                     static_cast<uint16_t*>(out), nope_dim, latent_dim);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return kvk::fail(KVK_ERR_DEVICE, "W_UK arrange launch: %s", hipGetErrorString(e));
  return KVK_OK;
}
