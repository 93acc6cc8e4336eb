// Query-aware token selection at prefill (the eviction composed with the cache
// configurations, KV-Kaizen §3.4; the paper's eviction implementations sum
// attention over a 32-query observation window, App. F.3).
//
// Per (sequence b, KV head h), from the prompt's keys K [n, D] and the queries of
// its last 32 positions (the G query heads of h, 32 each: R = 32 G rows):
//   importance(t) = sum over the R rows of softmax(scale q . k)(t), each window
//                   query attending causally (row of window slot w sees t <= n-32+w);
//   keep = the 32 window positions + the keep-32 prefix positions of largest
//          importance (ties to the lower position), in increasing order.
//
// Kernels (all sizes from the table; one call per anchor layer):
//   snap_scores_kernel<D, 0>: S = Q K^T on MFMA (bf16 in, fp32 out) over a
//       2048-token chunk per workgroup; per row the chunk's max and sum of 2^(s-max)
//       (online, rescaled only when the max moves).
//   snap_merge_kernel: per row (one wave), the chunks' (max, sum) merged into (M, 1/L).
//   snap_scores_kernel<D, 1>: S again, p = 2^(s - M) / L summed over the rows.
//   topk_*_kernel: radix select (12-, 10- and 9-bit digits of the fp32 pattern,
//       importance >= 0) of the threshold over slices of each stream's positions,
//       then an in-order pass that writes the kept positions already sorted.
// The keys are read twice from HBM; the queries sit in LDS.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "kvk_device.h"
#include "kvk_internal.h"

using namespace kvkd;

namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kWin = 32;      // observation window
constexpr int kChunk = 2048;  // tokens per workgroup in the score passes
constexpr int kMaxG = 8;      // query heads per KV head

struct SnapArgs {
  const uint16_t* k;  // [BH][n][D] bf16
  const uint16_t* q;  // [B][Hq][32][D] bf16
  float* part;        // [BH][P][R] x (max, sum)
  float* stats;       // [BH][R] x (M, 1/L)
  float* imp;         // [BH][n]
  int32_t* keep;      // [BH][keep_n]
  int32_t n, P, R, Hkv, Hq, keep_n;
  float scale_log2;
};

__device__ __forceinline__ f4 mfma_bf16(bf16x8 a, bf16x8 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// PASS 0: per-chunk row statistics.  PASS 1: importance of every token.
// Wave w of the workgroup takes token tiles of 16 at chunk offsets 16 w, 16 w + 64, ..
// S^T tile layout (A = 16 query rows, B = 16 tokens): lane (token i16, row group kg)
// holds rows 4 kg .. 4 kg + 3 of its token.
template <int D, int PASS, int G>
__global__ __launch_bounds__(256) void snap_scores_kernel(SnapArgs a) {
  constexpr int RT = 2 * G;  // row tiles of 16
  constexpr int R = 32 * G;  // window rows of the KV head
  constexpr int PQ = D + 8;  // LDS row pitch (bf16): consecutive rows 16 bytes apart in bank space
  extern __shared__ uint16_t qs[];  // [R][PQ], sized by the launch
  __shared__ float red[4][R][2];
  const int tid = threadIdx.x, lane = tid & 63, i16 = lane & 15, kg = lane >> 4;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int bh = blockIdx.y, p = blockIdx.x;
  const int b = bh / a.Hkv, h = bh % a.Hkv;
  const uint16_t* qb = a.q + (int64_t)(b * a.Hq + h * G) * kWin * D;
  for (int c = tid; c < R * (D / 8); c += 256) {
    const int r = c / (D / 8), o = 8 * (c % (D / 8));
    *reinterpret_cast<uint4*>(&qs[r * PQ + o]) = *reinterpret_cast<const uint4*>(qb + (int64_t)r * D + o);
  }
  __syncthreads();

  float m[RT][4], l[RT][4];  // PASS 0: running max / sum of 2^(s - max)
  float sm[RT][4], sl[RT][4];  // PASS 1: M and 1/L of the lane's rows
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if constexpr (PASS == 0) {
        m[rt][e] = -INFINITY;
        l[rt][e] = 0.0f;
      } else {
        const int r = 16 * rt + 4 * kg + e;
        const float* st = a.stats + ((int64_t)bh * R + r) * 2;
        sm[rt][e] = st[0];
        sl[rt][e] = st[1];
      }
    }

  const int t0 = p * kChunk, t1 = min(a.n, t0 + kChunk);
  const uint16_t* kb = a.k + (int64_t)bh * a.n * D;
  // The key operand of the next tile is loaded while the current one is computed.
  bf16x8 kn[D / 32];
  auto load_keys = [&](int t) {
#pragma unroll
    for (int j = 0; j < D / 32; ++j) {
      if (t < t1) kn[j] = *reinterpret_cast<const bf16x8*>(kb + (int64_t)t * D + 32 * j + 8 * kg);
      else kn[j] = bf16x8{};
    }
  };
  load_keys(t0 + 16 * wv + i16);
  for (int tt = t0 + 16 * wv; tt < t1; tt += 64) {
    const int t = tt + i16;
    bf16x8 kv[D / 32];
#pragma unroll
    for (int j = 0; j < D / 32; ++j) kv[j] = kn[j];
    load_keys(t + 64);
    float imp = 0.0f;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      {
        f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < D / 32; ++j) {
          const bf16x8 qa = *reinterpret_cast<const bf16x8*>(&qs[(16 * rt + i16) * PQ + 32 * j + 8 * kg]);
          acc = mfma_bf16(qa, kv[j], acc);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int w = (16 * rt + 4 * kg + e) & (kWin - 1);  // window slot of the row (rows are head-major)
          const bool vis = t < a.n && t <= a.n - kWin + w;
          const float s = acc[e] * a.scale_log2;
          if constexpr (PASS == 0) {
            if (vis) {
              if (s > m[rt][e]) {
                l[rt][e] *= __builtin_amdgcn_exp2f(m[rt][e] - s);
                m[rt][e] = s;
              }
              l[rt][e] += __builtin_amdgcn_exp2f(s - m[rt][e]);
            }
          } else {
            if (vis) imp += __builtin_amdgcn_exp2f(s - sm[rt][e]) * sl[rt][e];
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);  // one row tile's operands live at a time
    }
    if constexpr (PASS == 1) {
      imp = rows_sum(imp);  // over the four row groups
      if (kg == 0 && t < a.n) a.imp[(int64_t)bh * a.n + t] = imp;
    }
  }

  if constexpr (PASS == 0) {
    // over the 16 tokens of a row group (lanes i16), then over the 4 waves
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float M = max16(m[rt][e]);
          const float x = M == -INFINITY ? 0.0f : l[rt][e] * __builtin_amdgcn_exp2f(m[rt][e] - M);
          const float L = sum16(x);
          if (i16 == 0) {
            red[wv][16 * rt + 4 * kg + e][0] = M;
            red[wv][16 * rt + 4 * kg + e][1] = L;
          }
        }
      }
    }
    __syncthreads();
    if (tid < R) {
      float M = -INFINITY;
#pragma unroll
      for (int w = 0; w < 4; ++w) M = fmaxf(M, red[w][tid][0]);
      float L = 0.0f;
      if (M != -INFINITY) {
#pragma unroll
        for (int w = 0; w < 4; ++w)
          if (red[w][tid][0] != -INFINITY) L += red[w][tid][1] * __builtin_amdgcn_exp2f(red[w][tid][0] - M);
      }
      float* out = a.part + (((int64_t)bh * a.P + p) * R + tid) * 2;
      out[0] = M;
      out[1] = L;
    }
  }
}

// Per (b, h) and row: merge the chunks' (max, sum) into (M, 1/L).
__device__ __forceinline__ float wave_max64(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x = fmaxf(x, __shfl_xor(x, off));
  return x;
}
__device__ __forceinline__ float wave_sum64(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

// One wave per (stream, row): lane p merges chunks p, p + 64, ..., then the wave
// reduces (a reduction order fixed by the lane count, so results repeat exactly).
__global__ __launch_bounds__(256) void snap_merge_kernel(SnapArgs a) {
  const int bh = blockIdx.y, r = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (r >= a.R) return;
  const float* pp = a.part + (int64_t)bh * a.P * a.R * 2;
  float M = -INFINITY;
  for (int p = lane; p < a.P; p += 64) M = fmaxf(M, pp[((int64_t)p * a.R + r) * 2]);
  M = wave_max64(M);
  float L = 0.0f;
  for (int p = lane; p < a.P; p += 64) {
    const float mp = pp[((int64_t)p * a.R + r) * 2];
    if (mp != -INFINITY) L += pp[((int64_t)p * a.R + r) * 2 + 1] * __builtin_amdgcn_exp2f(mp - M);
  }
  L = wave_sum64(L);
  if (lane == 0) {
    float* st = a.stats + ((int64_t)bh * a.R + r) * 2;
    st[0] = M;
    st[1] = 1.0f / L;  // every row sees position 0, so L >= 1
  }
}

// Exclusive prefix sum over the 1024 threads of a workgroup (16 waves); total out.
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* wsum, uint32_t& total) {
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  uint32_t x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  if (lane == 63) wsum[wv] = x;
  __syncthreads();
  uint32_t before = 0, all = 0;
  for (int w = 0; w < 16; ++w) {
    const uint32_t s = wsum[w];
    if (w < wv) before += s;
    all += s;
  }
  __syncthreads();
  total = all;
  return before + x - v;
}

// Lanes of the wave below this one whose bit is set in the ballot.
__device__ __forceinline__ uint32_t lanes_below(uint64_t ballot, int lane) {
  return (uint32_t)__popcll(ballot & ((1ull << lane) - 1ull));
}

// Selection per stream (a (b, h) pair, or a sequence of an MLA layer): the keep - 32
// largest prefix importances (ties to the lower position) and the window, in
// increasing order.  The threshold is found by radix select over the fp32 pattern
// (importance >= 0, so patterns order as values): digits of 12, 10 and 9 bits below
// the sign.  The positions of a stream are cut into slices, one 1024-thread
// workgroup each, so that a launch spreads over the GPU: per digit one launch builds
// the histogram (in LDS per slice, then added into the stream's histogram in the
// workspace) and one picks the digit; then the slices count what they keep and write
// their positions at their offsets (each wave a contiguous sixteenth of its slice,
// ballots giving the ranks inside each 64-position step).
struct TopkArgs {
  const uint32_t* key;  // [S][n] fp32 patterns of the importances
  int32_t* keep;        // [S][keep_n]
  uint32_t* hist;       // [S][kTopkBins]: the histograms of digits 0, 1, 2
  uint32_t* state;      // [S][4][4]: (prefix, mask, remaining) before digit 0, 1, 2 and after 2
  uint32_t* cnt;        // [S][P][2]: positions above and at the threshold per slice
  int32_t n, keep_n, P, slice;
};

template <int DG>
struct Digit {
  static constexpr int SH = DG == 0 ? 19 : (DG == 1 ? 9 : 0);         // lowest bit
  static constexpr int NB = DG == 0 ? 4096 : (DG == 1 ? 1024 : 512);  // bins
  static constexpr int OFF = DG == 0 ? 0 : (DG == 1 ? 4096 : 5120);   // in the stream's histograms
};
constexpr int kTopkBins = 4096 + 1024 + 512;

// The stream's histograms cleared and its state set: no prefix yet, keep - 32 to find.
__global__ __launch_bounds__(256) void topk_init_kernel(TopkArgs a) {
  const int s = blockIdx.x;
  for (int i = threadIdx.x; i < kTopkBins; i += 256) a.hist[(int64_t)s * kTopkBins + i] = 0u;
  if (threadIdx.x < 4) a.state[16 * s + threadIdx.x] = threadIdx.x == 2 ? (uint32_t)(a.keep_n - kWin) : 0u;
}

// Digit DG of the threshold, from the state before it and the finished histogram of
// the digit: over the digits in descending order, four per thread, the thread whose
// range holds the remaining-th largest key fixes it.  Every workgroup of a launch
// computes it alike; the state after the digit comes back in st (shared), and the
// first slice's workgroup stores it for the launches that follow.
template <int DG>
__device__ __forceinline__ void topk_pick(const TopkArgs& a, int s, int tid, uint32_t* wsum, uint32_t* st) {
  constexpr int SH = Digit<DG>::SH, NB = Digit<DG>::NB;
  const uint32_t* g = a.hist + (int64_t)s * kTopkBins + Digit<DG>::OFF;
  const uint32_t* prev = a.state + 16 * s + 4 * DG;
  const uint32_t prefix = prev[0], mask = prev[1], remaining = prev[2];
  if (tid == 0) {  // unchanged unless a thread owns the digit (one always does)
    st[0] = prefix;
    st[1] = mask | ((uint32_t)(NB - 1) << SH);
    st[2] = remaining;
  }
  const int top = NB - 1 - 4 * tid;
  uint32_t c[4] = {0u, 0u, 0u, 0u}, c4 = 0u;
  if (top >= 0)
    for (int j = 0; j < 4; ++j) {
      c[j] = g[top - j];
      c4 += c[j];
    }
  uint32_t tot;
  const uint32_t above = block_exclusive_scan(c4, wsum, tot);  // (its barriers order st's first write)
  if (top >= 0 && above < remaining && above + c4 >= remaining) {
    uint32_t cum = above;
    for (int j = 0; j < 4; ++j) {
      if (cum + c[j] >= remaining) {
        st[0] = prefix | ((uint32_t)(top - j) << SH);
        st[2] = remaining - cum;
        break;
      }
      cum += c[j];
    }
  }
  __syncthreads();
  if (blockIdx.x == 0 && tid < 3) a.state[16 * s + 4 * (DG + 1) + tid] = st[tid];
}

// Histogram of digit DG over one slice, for the keys that carry the prefix so far
// (for DG > 0 fixed here first from the previous digit's histogram).
template <int DG>
__global__ __launch_bounds__(1024) void topk_hist_kernel(TopkArgs a) {
  constexpr int SH = Digit<DG>::SH, NB = Digit<DG>::NB;
  __shared__ uint32_t h[NB];
  __shared__ uint32_t wsum[16], st[4];
  const int s = blockIdx.y, tid = threadIdx.x;
  const int np = a.n - kWin;
  uint32_t prefix = 0u, mask = 0u;
  if constexpr (DG > 0) {
    topk_pick<DG - 1>(a, s, tid, wsum, st);
    prefix = st[0];
    mask = st[1];
  }
  for (int i = tid; i < NB; i += 1024) h[i] = 0u;
  __syncthreads();
  const uint32_t* key = a.key + (int64_t)s * a.n;
  const int i0 = blockIdx.x * a.slice, i1 = min(np, i0 + a.slice);
  for (int i = i0 + tid; i < i1; i += 1024) {
    const uint32_t u = key[i];
    if ((u & mask) == prefix) atomicAdd(&h[(u >> SH) & (uint32_t)(NB - 1)], 1u);
  }
  __syncthreads();
  uint32_t* g = a.hist + (int64_t)s * kTopkBins + Digit<DG>::OFF;
  for (int i = tid; i < NB; i += 1024)
    if (h[i] != 0u) atomicAdd(&g[i], h[i]);
}

// Per slice: the last digit fixed (the threshold pattern and how many keys at it
// are kept), then the positions above the pattern and at it.
__global__ __launch_bounds__(1024) void topk_count_kernel(TopkArgs a) {
  __shared__ uint32_t wsum[16], st[4];
  const int s = blockIdx.y, tid = threadIdx.x;
  const int np = a.n - kWin;
  topk_pick<2>(a, s, tid, wsum, st);
  const uint32_t prefix = st[0];
  const uint32_t* key = a.key + (int64_t)s * a.n;
  const int i0 = blockIdx.x * a.slice, i1 = min(np, i0 + a.slice);
  uint32_t n_gt = 0u, n_eq = 0u;
  for (int i = i0 + tid; i < i1; i += 1024) {
    const uint32_t u = key[i];
    n_gt += u > prefix ? 1u : 0u;
    n_eq += u == prefix ? 1u : 0u;
  }
  uint32_t tot_gt, tot_eq;
  block_exclusive_scan(n_gt, wsum, tot_gt);
  block_exclusive_scan(n_eq, wsum, tot_eq);
  if (tid == 0) {
    uint32_t* c = a.cnt + ((int64_t)s * a.P + blockIdx.x) * 2;
    c[0] = tot_gt;
    c[1] = tot_eq;
  }
}

// The slice's kept positions at its offset: every position above the threshold
// pattern, and those at it while fewer than `remaining` came before (position order).
// Slice 0 also writes the window.  select: false when nothing is selected (keep =
// the window).
__global__ __launch_bounds__(1024) void topk_write_kernel(TopkArgs a, int select) {
  __shared__ uint32_t wgt[16], weq[16];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int s = blockIdx.y;
  const int np = a.n - kWin, k = a.keep_n - kWin;
  int32_t* out = a.keep + (int64_t)s * a.keep_n;
  if (select) {
    const uint32_t prefix = a.state[16 * s + 12], remaining = a.state[16 * s + 14];  // after digit 2
    const uint32_t* key = a.key + (int64_t)s * a.n;
    uint32_t gt_slices = 0u, eq_slices = 0u;  // the slices before this one
    for (int j = 0; j < (int)blockIdx.x; ++j) {
      gt_slices += a.cnt[((int64_t)s * a.P + j) * 2];
      eq_slices += a.cnt[((int64_t)s * a.P + j) * 2 + 1];
    }
    const int i0 = blockIdx.x * a.slice, i1 = min(np, i0 + a.slice);
    const int seg = (i1 - i0 + 15) / 16;
    const int r0 = min(i1, i0 + wv * seg), r1 = min(i1, r0 + seg);
    uint32_t n_gt = 0u, n_eq = 0u;
    for (int base = r0; base < r1; base += 64) {
      const int i = base + lane;
      const uint32_t u = i < r1 ? key[i] : 0u;
      n_gt += (uint32_t)__popcll(__ballot(i < r1 && u > prefix));
      n_eq += (uint32_t)__popcll(__ballot(i < r1 && u == prefix));
    }
    if (lane == 0) {
      wgt[wv] = n_gt;
      weq[wv] = n_eq;
    }
    __syncthreads();
    uint32_t gt_before = gt_slices, eq_before = eq_slices;
    for (int w = 0; w < wv; ++w) {
      gt_before += wgt[w];
      eq_before += weq[w];
    }
    uint32_t off = gt_before + min(eq_before, remaining), eq_seen = eq_before;
    for (int base = r0; base < r1; base += 64) {
      const int i = base + lane;
      const bool in = i < r1;
      const uint32_t u = in ? key[i] : 0u;
      const bool eq = in && u == prefix;
      const uint64_t beq = __ballot(eq);
      const bool take = in && (u > prefix || (eq && eq_seen + lanes_below(beq, lane) < remaining));
      const uint64_t bt = __ballot(take);
      const uint32_t o = off + lanes_below(bt, lane);
      if (take && o < (uint32_t)k) out[o] = i;  // o < k holds by construction; kept as a guard
      off += (uint32_t)__popcll(bt);
      eq_seen += (uint32_t)__popcll(beq);
    }
  }
  if (blockIdx.x == 0)
    for (int i = tid; i < kWin; i += 1024) out[k + i] = np + i;
}

// ---------------------------------------------------------------------------
// MLA layers (one keep list per sequence: the heads share the latent).  Rows of a
// sequence are (window slot w, head h), row index w Hp + h over the padded head
// count Hp; the absorbed window queries q~ = W_UK[h]^T q_nope (full latent width
// r, prescaled by scale log2 e, fp16) and the RoPE part, [B][32][Hp][r + d_R], come
// from the absorption kernel.  Head h's score of position t is then
// q~ . c_t + q_rope . k^R_t; padding heads (h >= Hq) take no part.
// ---------------------------------------------------------------------------

constexpr int kMlaChunk = 256;  // tokens per workgroup in the MLA score passes
// The MLA score passes' workgroups: 8 waves, each holding the query fragments of
// two 16-row tiles up to r = 512 (one above, whose fragments take 136 registers), so
// that the chunk's latent, converted to fp16 once per workgroup, serves 256 (128)
// rows, and each LDS read of it feeds two score products.
constexpr int kMlaWaves = 8;
constexpr int snap_mla_row_tiles(int r) { return r <= 512 ? 2 : 1; }

struct SnapMlaArgs {
  const uint16_t* lat;   // [B][n][r] bf16 latent (full width)
  const uint16_t* rope;  // [B][n][64] bf16 positional keys
  const _Float16* q;     // [B][32][Hp][r + 64] absorbed window queries
  float* part;           // [B][RB][P][rpb] x (max, sum)
  float* stats;          // [B][32 Hp] x (M, 1/L)
  float* ipart;          // [B][RB][n] importance of each row block
  float* imp;            // [B][n]
  int32_t n, P, RB, Hq, Hp, r;
  int32_t rpb;           // rows per block (16 per wave)
};

__device__ __forceinline__ f4 mfma_f16(half8 a, half8 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// One workgroup per (256-token chunk, row block, sequence); wave w holds the fp16
// fragments of its RT 16-row tiles (rows 16 (RT w + t) .. + 15 of the block, B
// operands) for the whole chunk.  Per 32 tokens the chunk's latent and positional
// keys are staged in LDS as fp16 rows (pitch W + 8 halfs: 16 consecutive rows start
// 16 distinct 4-bank windows apart; the next step's are loaded meanwhile) and each
// wave scores both 16-token tiles, every A operand read from LDS once for its RT row
// tiles: lane (i16, kg) gets tokens 4 kg .. + 3 of row i16 of each tile.  (Reading
// the tile is what bounds the passes: each wave reads all of it, so more rows per
// wave means fewer reads per score.)
// PASS 0: per row the chunk's max and sum of 2^(s - max).  PASS 1: per token the sum
// over the block's rows of 2^(s - M) / L.
template <int NK, int PASS, int WV, int RT>
__global__ __launch_bounds__(64 * WV) void snap_mla_scores_kernel(SnapMlaArgs a) {
  constexpr int W = 32 * NK, PT = W + 8, NT = 64 * WV;
  __shared__ __attribute__((aligned(16))) _Float16 tile[32 * PT];
  __shared__ float red[WV][32];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, i16 = lane & 15, kg = lane >> 4;
  const int p = blockIdx.x, rb = blockIdx.y, b = blockIdx.z;
  int lastvis[RT];  // the row's window query sees t <= lastvis
  bool valid[RT];
  half8 qf[RT][NK];
  float m[RT], l[RT], sM[RT], sL[RT];
#pragma unroll
  for (int r = 0; r < RT; ++r) {
    const int row = 16 * RT * WV * rb + 16 * (RT * wv + r) + i16;  // w Hp + h
    const int w = row / a.Hp, h = row - w * a.Hp;
    valid[r] = h < a.Hq;
    lastvis[r] = a.n - kWin + w;
    const _Float16* qr = a.q + ((int64_t)b * kWin * a.Hp + row) * W + 8 * kg;
#pragma unroll
    for (int j = 0; j < NK; ++j) qf[r][j] = *reinterpret_cast<const half8*>(qr + 32 * j);
    m[r] = -INFINITY;
    l[r] = sM[r] = sL[r] = 0.0f;
    if constexpr (PASS == 1) {
      if (valid[r]) {
        sM[r] = a.stats[((int64_t)b * kWin * a.Hp + row) * 2];
        sL[r] = a.stats[((int64_t)b * kWin * a.Hp + row) * 2 + 1];
      }
    }
  }
  const int t0 = p * kMlaChunk, t1 = min(a.n, t0 + kMlaChunk);
  // Each thread moves CPT 8-channel pieces of a 32-token step; the next step's are
  // loaded while the current one is scored (register double buffering).
  constexpr int NC = 32 * (W / 8), CPT = (NC + NT - 1) / NT;
  u4v pre[CPT];
  auto fetch = [&](int tb) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = tid + i * NT;
      const int tr = c / (W / 8), c8 = 8 * (c - tr * (W / 8));
      const int t = tb + tr;
      pre[i] = u4v{0u, 0u, 0u, 0u};
      if (c < NC && t < t1)
        pre[i] = c8 < a.r ? *reinterpret_cast<const u4v*>(a.lat + ((int64_t)b * a.n + t) * a.r + c8)
                          : *reinterpret_cast<const u4v*>(a.rope + ((int64_t)b * a.n + t) * 64 + (c8 - a.r));
    }
  };
  fetch(t0);
  for (int tb = t0; tb < t1; tb += 32) {
    __syncthreads();  // the tile (and red) are free
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = tid + i * NT;
      if (c < NC) {
        const int tr = c / (W / 8), c8 = 8 * (c - tr * (W / 8));
        half8 x;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          x[2 * e] = (_Float16)__uint_as_float(pre[i][e] << 16);
          x[2 * e + 1] = (_Float16)__uint_as_float(pre[i][e] & 0xFFFF0000u);
        }
        *reinterpret_cast<half8*>(tile + tr * PT + c8) = x;
      }
    }
    if (tb + 32 < t1) fetch(tb + 32);
    __syncthreads();
    float x[RT][2][4];  // scores (PASS 0, masked) or probabilities (PASS 1)
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
      f4 acc[RT];
#pragma unroll
      for (int r = 0; r < RT; ++r) acc[r] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < NK; ++j) {
        const half8 av = *reinterpret_cast<const half8*>(tile + (16 * tt + i16) * PT + 32 * j + 8 * kg);
#pragma unroll
        for (int r = 0; r < RT; ++r) acc[r] = mfma_f16(av, qf[r][j], acc[r]);
      }
#pragma unroll
      for (int r = 0; r < RT; ++r)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int t = tb + 16 * tt + 4 * kg + e;
          const bool vis = valid[r] && t < t1 && t <= lastvis[r];
          if constexpr (PASS == 0) x[r][tt][e] = vis ? acc[r][e] : -INFINITY;
          else x[r][tt][e] = vis ? __builtin_amdgcn_exp2f(acc[r][e] - sM[r]) * sL[r] : 0.0f;
        }
    }
    if constexpr (PASS == 0) {  // online max and sum over the step's 8 tokens of each row
#pragma unroll
      for (int r = 0; r < RT; ++r) {
        float mx = x[r][0][0];
#pragma unroll
        for (int k = 1; k < 8; ++k) mx = fmaxf(mx, x[r][k >> 2][k & 3]);
        if (mx > m[r]) {
          l[r] *= __builtin_amdgcn_exp2f(m[r] - mx);
          m[r] = mx;
        }
        if (m[r] != -INFINITY) {
#pragma unroll
          for (int k = 0; k < 8; ++k) l[r] += __builtin_amdgcn_exp2f(x[r][k >> 2][k & 3] - m[r]);
        }
      }
    } else {
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float sum = 0.0f;  // over the wave's rows, tile by tile
#pragma unroll
          for (int r = 0; r < RT; ++r) sum += sum16(x[r][tt][e]);
          if (i16 == 0) red[wv][16 * tt + 4 * kg + e] = sum;
        }
      __syncthreads();
      if (tid < 32 && tb + tid < t1) {
        float sum = 0.0f;  // the waves' sums in wave order
#pragma unroll
        for (int v = 0; v < WV; ++v) sum += red[v][tid];
        a.ipart[((int64_t)b * a.RB + rb) * a.n + tb + tid] = sum;
      }
    }
  }
  if constexpr (PASS == 0) {  // the row's four token groups (lanes i16 + 16 kg)
#pragma unroll
    for (int r = 0; r < RT; ++r) {
      const float M = rows_max(m[r]);
      const float L = rows_sum(M == -INFINITY ? 0.0f : l[r] * __builtin_amdgcn_exp2f(m[r] - M));
      if (kg == 0) {
        float* out = a.part + (((int64_t)b * a.RB + rb) * a.P + p) * (2 * a.rpb) + 2 * (16 * (RT * wv + r) + i16);
        out[0] = M;
        out[1] = L;
      }
    }
  }
}

// Per (sequence, row): the chunks' (max, sum) merged into (M, 1/L).
// One wave per (sequence, row), as snap_merge_kernel.
__global__ __launch_bounds__(256) void snap_mla_merge_kernel(SnapMlaArgs a) {
  const int b = blockIdx.y, row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= kWin * a.Hp) return;
  const int rb = row / a.rpb, rr = row - rb * a.rpb;
  const int64_t ps = 2 * a.rpb;  // floats per (row block, chunk)
  const float* pp = a.part + ((int64_t)b * a.RB + rb) * a.P * ps + 2 * rr;
  float M = -INFINITY;
  for (int p = lane; p < a.P; p += 64) M = fmaxf(M, pp[(int64_t)p * ps]);
  M = wave_max64(M);
  float L = 0.0f;
  for (int p = lane; p < a.P; p += 64) {
    const float mp = pp[(int64_t)p * ps];
    if (mp != -INFINITY) L += pp[(int64_t)p * ps + 1] * __builtin_amdgcn_exp2f(mp - M);
  }
  L = wave_sum64(L);
  if (lane == 0) {
    float* st = a.stats + ((int64_t)b * kWin * a.Hp + row) * 2;
    st[0] = M;
    st[1] = L > 0.0f ? 1.0f / L : 0.0f;  // a padding head's row has no mass
  }
}

// importance[b][t] = the row blocks' partial sums, added in block order.
__global__ __launch_bounds__(256) void snap_mla_reduce_kernel(SnapMlaArgs a) {
  const int b = blockIdx.y, t = blockIdx.x * 256 + threadIdx.x;
  if (t >= a.n) return;
  const float* ip = a.ipart + (int64_t)b * a.RB * a.n + t;
  float s = 0.0f;
  for (int rb = 0; rb < a.RB; ++rb) s += ip[(int64_t)rb * a.n];
  a.imp[(int64_t)b * a.n + t] = s;
}

}  // namespace

using namespace kvk;

namespace {

struct SnapSizes {
  int64_t part, stats, imp;  // floats
  int32_t P, R;
};

// The selection's slices and scratch for S streams of n positions: slices of at least
// 4096 positions, as many as keep about 512 workgroups busy.
struct TopkSizes {
  int32_t P, slice;
  int64_t hist, state, cnt;  // bytes
};

TopkSizes topk_sizes(int64_t S, int32_t n_tokens) {
  TopkSizes z;
  const int32_t np = n_tokens - kWin > 0 ? n_tokens - kWin : 0;
  const int64_t by_size = (np + 4095) / 4096, by_count = (512 + S - 1) / S;
  z.P = (int32_t)std::max<int64_t>(1, std::min(by_size, by_count));
  z.slice = ((np + z.P - 1) / z.P + 63) / 64 * 64;
  if (z.slice == 0) z.slice = 64;
  z.hist = round256(S * kTopkBins * 4);
  z.state = round256(S * 16 * 4);
  z.cnt = round256(S * z.P * 2 * 4);
  return z;
}

// The selection over S streams of importances (keys) into keep lists; scratch: the
// topk_sizes bytes at `w`.
void launch_topk(const float* imp, int32_t* keep, int64_t S, int32_t n_tokens, int32_t keep_n, uint8_t* w,
                 hipStream_t stream) {
  const TopkSizes z = topk_sizes(S, n_tokens);
  TopkArgs t;
  t.key = reinterpret_cast<const uint32_t*>(imp);
  t.keep = keep;
  t.hist = reinterpret_cast<uint32_t*>(w);
  t.state = reinterpret_cast<uint32_t*>(w + z.hist);
  t.cnt = reinterpret_cast<uint32_t*>(w + z.hist + z.state);
  t.n = n_tokens;
  t.keep_n = keep_n;
  t.P = z.P;
  t.slice = z.slice;
  const dim3 gs((unsigned)z.P, (unsigned)S), b1024(1024);
  const bool select = keep_n - kWin > 0;
  if (select) {
    hipLaunchKernelGGL(topk_init_kernel, dim3((unsigned)S), dim3(256), 0, stream, t);
    hipLaunchKernelGGL(topk_hist_kernel<0>, gs, b1024, 0, stream, t);
    hipLaunchKernelGGL(topk_hist_kernel<1>, gs, b1024, 0, stream, t);  // digit 0 fixed first
    hipLaunchKernelGGL(topk_hist_kernel<2>, gs, b1024, 0, stream, t);  // digit 1 fixed first
    hipLaunchKernelGGL(topk_count_kernel, gs, b1024, 0, stream, t);    // digit 2 fixed first
  }
  hipLaunchKernelGGL(topk_write_kernel, gs, b1024, 0, stream, t, select ? 1 : 0);
}

SnapSizes snap_sizes(const kvk_table* t, int32_t n_tokens) {
  const kvk_dims& d = t->d;
  SnapSizes s;
  s.P = (n_tokens + kChunk - 1) / kChunk;
  s.R = kWin * (d.n_q_heads / d.n_kv_heads);
  const int64_t bh = (int64_t)d.batch * d.n_kv_heads;
  s.part = bh * s.P * s.R * 2;
  s.stats = bh * s.R * 2;
  s.imp = bh * n_tokens;
  return s;
}

template <int PASS>
void launch_scores(int D, int G, dim3 gs, size_t lds, hipStream_t stream, const SnapArgs& a) {
#define KVK_SNAP(DD, GG) \
  if (D == DD && G == GG) { \
    hipLaunchKernelGGL((snap_scores_kernel<DD, PASS, GG>), gs, dim3(256), lds, stream, a); \
    return; \
  }
  KVK_SNAP(128, 1) KVK_SNAP(128, 2) KVK_SNAP(128, 3) KVK_SNAP(128, 4)
  KVK_SNAP(128, 5) KVK_SNAP(128, 6) KVK_SNAP(128, 7) KVK_SNAP(128, 8)
  KVK_SNAP(64, 1) KVK_SNAP(64, 2) KVK_SNAP(64, 3) KVK_SNAP(64, 4)
  KVK_SNAP(64, 5) KVK_SNAP(64, 6) KVK_SNAP(64, 7) KVK_SNAP(64, 8)
#undef KVK_SNAP
}

struct SnapMlaSizes {
  int64_t q, part, stats, ipart, imp;  // bytes
  int32_t P, RB, Hp, rpb;
};

SnapMlaSizes snap_mla_sizes(const kvk_table* t, int32_t n_tokens) {
  const kvk_dims& d = t->d;
  SnapMlaSizes s;
  s.Hp = mla_heads_padded(d.n_q_heads);
  s.P = (n_tokens + kMlaChunk - 1) / kMlaChunk;
  s.rpb = 16 * kMlaWaves * snap_mla_row_tiles(d.latent_dim);
  s.RB = kWin * s.Hp / s.rpb;  // 32 Hp is a multiple of 512
  s.q = round256((int64_t)d.batch * kWin * s.Hp * (d.latent_dim + d.rope_dim) * 2);
  s.part = round256((int64_t)d.batch * s.RB * s.P * 2 * s.rpb * 4);
  s.stats = round256((int64_t)d.batch * kWin * s.Hp * 2 * 4);
  s.ipart = round256((int64_t)d.batch * s.RB * n_tokens * 4);
  s.imp = round256((int64_t)d.batch * n_tokens * 4);
  return s;
}

kvk_status snap_check_common(const kvk_table* t, int32_t n_tokens) {
  const kvk_dims& d = t->d;
  if (d.keep_tokens < kWin)
    return fail(KVK_ERR_INVALID, "snapkv: the table must evict with keep_tokens >= %d (has %d)", kWin,
                d.keep_tokens);
  if (n_tokens < d.keep_tokens || n_tokens > d.max_tokens)
    return fail(KVK_ERR_INVALID, "snapkv: n_tokens %d outside keep_tokens..max_tokens (%d..%d)", n_tokens,
                d.keep_tokens, d.max_tokens);
  return KVK_OK;
}

kvk_status snap_mla_check(const kvk_table* t, int32_t n_tokens) {
  if (!t) return fail(KVK_ERR_INVALID, "snapkv: NULL table");
  const kvk_dims& d = t->d;
  if (d.kind != KVK_MLA) return fail(KVK_ERR_INVALID, "kvk_snapkv_select_mla: an MLA table is required");
  if (d.latent_dim != 256 && d.latent_dim != 512 && d.latent_dim != 768 && d.latent_dim != 1024)
    return fail(KVK_ERR_UNSUPPORTED, "kvk_snapkv_select_mla: latent_dim %d (256, 512, 768 or 1024)", d.latent_dim);
  return snap_check_common(t, n_tokens);
}

kvk_status snap_check(const kvk_table* t, int32_t n_tokens) {
  if (!t) return fail(KVK_ERR_INVALID, "snapkv: NULL table");
  const kvk_dims& d = t->d;
  if (d.kind != KVK_GQA) return fail(KVK_ERR_UNSUPPORTED, "kvk_snapkv_select: GQA tables (MLA: kvk_snapkv_select_mla)");
  if (d.keep_tokens < kWin)
    return fail(KVK_ERR_INVALID, "snapkv: the table must evict with keep_tokens >= %d (has %d)", kWin,
                d.keep_tokens);
  if (n_tokens < d.keep_tokens || n_tokens > d.max_tokens)
    return fail(KVK_ERR_INVALID, "snapkv: n_tokens %d outside keep_tokens..max_tokens (%d..%d)", n_tokens,
                d.keep_tokens, d.max_tokens);
  if (d.n_q_heads / d.n_kv_heads > kMaxG)
    return fail(KVK_ERR_UNSUPPORTED, "snapkv: at most %d query heads per KV head", kMaxG);
  if (d.head_dim != 64 && d.head_dim != 128) return fail(KVK_ERR_UNSUPPORTED, "snapkv: head_dim %d", d.head_dim);
  return KVK_OK;
}

}  // namespace

extern "C" kvk_status kvk_snapkv_workspace_bytes(const kvk_table* t, int32_t n_tokens, size_t* out) {
  if (t && t->d.kind == KVK_MLA) {
    const kvk_status st = snap_mla_check(t, n_tokens);
    if (st != KVK_OK) return st;
    if (!out) return fail(KVK_ERR_INVALID, "snapkv: NULL output");
    const SnapMlaSizes s = snap_mla_sizes(t, n_tokens);
    const TopkSizes z = topk_sizes(t->d.batch, n_tokens);
    *out = (size_t)(s.q + s.part + s.stats + s.ipart + s.imp + z.hist + z.state + z.cnt);
    return KVK_OK;
  }
  const kvk_status st = snap_check(t, n_tokens);
  if (st != KVK_OK) return st;
  if (!out) return fail(KVK_ERR_INVALID, "snapkv: NULL output");
  const SnapSizes s = snap_sizes(t, n_tokens);
  const TopkSizes z = topk_sizes((int64_t)t->d.batch * t->d.n_kv_heads, n_tokens);
  *out = (size_t)(round256(s.part * 4) + round256(s.stats * 4) + round256(s.imp * 4) + z.hist + z.state + z.cnt);
  return KVK_OK;
}

extern "C" kvk_status kvk_snapkv_select(const kvk_table* t, int32_t layer, const void* k, const void* q_obs,
                                        int32_t in_dtype, int32_t n_tokens, float scale, int32_t* keep_out,
                                        float* importance_out, void* workspace, size_t ws_bytes,
                                        hipStream_t stream) {
  kvk_status st = snap_check(t, n_tokens);
  if (st != KVK_OK) return st;
  const kvk_dims& d = t->d;
  if (layer < 0 || layer >= d.n_layers) return fail(KVK_ERR_INVALID, "layer %d out of range", layer);
  // an inheriting layer stores nothing to select from (per-sequence plans: every
  // sequence is scored; the write uses the lists of the sequences that store)
  if (t->seq.empty() && t->plan[layer].inherit) return KVK_OK;
  if (!k || !q_obs || !keep_out || !workspace) return fail(KVK_ERR_INVALID, "snapkv: NULL buffer");
  if (in_dtype != KVK_BF16) return fail(KVK_ERR_UNSUPPORTED, "snapkv: keys and queries must be bf16");
  if (!(scale == scale)) return fail(KVK_ERR_INVALID, "snapkv: scale is NaN");
  if ((reinterpret_cast<uintptr_t>(k) & 15) || (reinterpret_cast<uintptr_t>(q_obs) & 15) ||
      (reinterpret_cast<uintptr_t>(keep_out) & 3) || (reinterpret_cast<uintptr_t>(importance_out) & 3) ||
      (reinterpret_cast<uintptr_t>(workspace) & 255))
    return fail(KVK_ERR_INVALID, "snapkv: misaligned buffer (k/q 16 B, keep/importance 4 B, workspace 256 B)");
  size_t need = 0;
  kvk_snapkv_workspace_bytes(t, n_tokens, &need);
  if (need > ws_bytes) return fail(KVK_ERR_BUFFER, "snapkv: workspace %zu bytes < %zu needed", ws_bytes, need);
  const SnapSizes s = snap_sizes(t, n_tokens);
  const int64_t bh = (int64_t)d.batch * d.n_kv_heads;
  if (bh > 65535 || s.P > 0x7fffffff) return fail(KVK_ERR_UNSUPPORTED, "snapkv: grid too large");
  if (kvk_status st2 = check_gpu_buffers({k, q_obs, keep_out, importance_out, workspace}, "kvk_snapkv_select"))
    return st2;
  SnapArgs a;
  a.k = static_cast<const uint16_t*>(k);
  a.q = static_cast<const uint16_t*>(q_obs);
  uint8_t* w = static_cast<uint8_t*>(workspace);
  a.part = reinterpret_cast<float*>(w);
  a.stats = reinterpret_cast<float*>(w + round256(s.part * 4));
  a.imp = importance_out ? importance_out : reinterpret_cast<float*>(w + round256(s.part * 4) + round256(s.stats * 4));
  a.keep = keep_out;
  a.n = n_tokens;
  a.P = s.P;
  a.R = s.R;
  a.Hkv = d.n_kv_heads;
  a.Hq = d.n_q_heads;
  a.keep_n = d.keep_tokens;
  a.scale_log2 = scale * kLog2e;
  const dim3 gs((unsigned)s.P, (unsigned)bh), b256(256);
  const size_t lds_q = (size_t)s.R * (d.head_dim + 8) * sizeof(uint16_t);  // the window queries
  const int G = d.n_q_heads / d.n_kv_heads;
  launch_scores<0>(d.head_dim, G, gs, lds_q, stream, a);
  hipLaunchKernelGGL(snap_merge_kernel, dim3((unsigned)((s.R + 3) / 4), (unsigned)bh), b256, 0, stream, a);
  launch_scores<1>(d.head_dim, G, gs, lds_q, stream, a);
  launch_topk(a.imp, keep_out, bh, n_tokens, d.keep_tokens,
              w + round256(s.part * 4) + round256(s.stats * 4) + round256(s.imp * 4), stream);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(KVK_ERR_DEVICE, "snapkv launch: %s", hipGetErrorString(e));
  return KVK_OK;
}

extern "C" kvk_status kvk_snapkv_select_mla(const kvk_table* t, int32_t layer, const void* latent,
                                            const void* k_rope, const void* q_obs, const void* w_uk,
                                            int32_t n_tokens, float scale, int32_t* keep_out,
                                            float* importance_out, void* workspace, size_t ws_bytes,
                                            hipStream_t stream) {
  kvk_status st = snap_mla_check(t, n_tokens);
  if (st != KVK_OK) return st;
  const kvk_dims& d = t->d;
  if (layer < 0 || layer >= d.n_layers) return fail(KVK_ERR_INVALID, "layer %d out of range", layer);
  if (t->seq.empty() && t->plan[layer].inherit) return KVK_OK;  // nothing stored to select from
  if (!w_uk && t->mla_w_uk)
    w_uk = static_cast<const uint8_t*>(t->mla_w_uk) + (int64_t)layer * d.n_q_heads * d.latent_dim * d.nope_dim * 2;
  if (!latent || !k_rope || !q_obs || !w_uk || !keep_out || !workspace)
    return fail(KVK_ERR_INVALID, "kvk_snapkv_select_mla: NULL buffer (w_uk: passed or attached)");
  if (!(scale == scale)) return fail(KVK_ERR_INVALID, "snapkv: scale is NaN");
  if ((reinterpret_cast<uintptr_t>(latent) & 15) || (reinterpret_cast<uintptr_t>(k_rope) & 15) ||
      (reinterpret_cast<uintptr_t>(q_obs) & 15) || (reinterpret_cast<uintptr_t>(w_uk) & 15) ||
      (reinterpret_cast<uintptr_t>(keep_out) & 3) || (reinterpret_cast<uintptr_t>(importance_out) & 3) ||
      (reinterpret_cast<uintptr_t>(workspace) & 255))
    return fail(KVK_ERR_INVALID, "snapkv: misaligned buffer (inputs 16 B, keep/importance 4 B, workspace 256 B)");
  size_t need = 0;
  kvk_snapkv_workspace_bytes(t, n_tokens, &need);
  if (need > ws_bytes) return fail(KVK_ERR_BUFFER, "snapkv: workspace %zu bytes < %zu needed", ws_bytes, need);
  const SnapMlaSizes s = snap_mla_sizes(t, n_tokens);
  if (d.batch > 65535 || s.P > 65535 || s.RB > 65535) return fail(KVK_ERR_UNSUPPORTED, "snapkv: grid too large");
  if (kvk_status st2 = check_gpu_buffers({latent, k_rope, q_obs, w_uk, keep_out, importance_out, workspace},
                                         "kvk_snapkv_select_mla"))
    return st2;
  uint8_t* wsb = static_cast<uint8_t*>(workspace);
  // the absorbed window queries: the B x 32 window positions as rows of the absorption
  st = mla_absorb_rows(t, q_obs, d.batch * kWin, w_uk, wsb, scale, stream);
  if (st != KVK_OK) return st;
  SnapMlaArgs a;
  a.lat = static_cast<const uint16_t*>(latent);
  a.rope = static_cast<const uint16_t*>(k_rope);
  a.q = reinterpret_cast<const _Float16*>(wsb);
  a.part = reinterpret_cast<float*>(wsb + s.q);
  a.stats = reinterpret_cast<float*>(wsb + s.q + s.part);
  a.ipart = reinterpret_cast<float*>(wsb + s.q + s.part + s.stats);
  a.imp = importance_out ? importance_out : reinterpret_cast<float*>(wsb + s.q + s.part + s.stats + s.ipart);
  a.n = n_tokens;
  a.P = s.P;
  a.RB = s.RB;
  a.rpb = s.rpb;
  a.Hq = d.n_q_heads;
  a.Hp = s.Hp;
  a.r = d.latent_dim;
  const dim3 gs((unsigned)s.P, (unsigned)s.RB, (unsigned)d.batch), b256(256), bw(64 * kMlaWaves);
  const dim3 gm((unsigned)((kWin * s.Hp + 3) / 4), (unsigned)d.batch);  // a wave per row
  const dim3 gr((unsigned)((n_tokens + 255) / 256), (unsigned)d.batch);
#define KVK_SNAP_MLA(PASS)                                                                                  \
  switch (d.latent_dim) {                                                                                   \
    case 256: hipLaunchKernelGGL((snap_mla_scores_kernel<10, PASS, kMlaWaves, 2>), gs, bw, 0, stream, a); break; \
    case 512: hipLaunchKernelGGL((snap_mla_scores_kernel<18, PASS, kMlaWaves, 2>), gs, bw, 0, stream, a); break; \
    case 768: hipLaunchKernelGGL((snap_mla_scores_kernel<26, PASS, kMlaWaves, 1>), gs, bw, 0, stream, a); break; \
    default: hipLaunchKernelGGL((snap_mla_scores_kernel<34, PASS, kMlaWaves, 1>), gs, bw, 0, stream, a); break;  \
  }
  KVK_SNAP_MLA(0)
  hipLaunchKernelGGL(snap_mla_merge_kernel, gm, b256, 0, stream, a);
  KVK_SNAP_MLA(1)
#undef KVK_SNAP_MLA
  hipLaunchKernelGGL(snap_mla_reduce_kernel, gr, b256, 0, stream, a);
  // the selection, one stream per sequence
  launch_topk(a.imp, keep_out, d.batch, n_tokens, d.keep_tokens, wsb + s.q + s.part + s.stats + s.ipart + s.imp,
              stream);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(KVK_ERR_DEVICE, "snapkv (MLA) launch: %s", hipGetErrorString(e));
  return KVK_OK;
}
