// Prefill write of a layer's compressed cache (W1) and the test-only dequantiser.
//
// An anchor layer stores, per (sequence, KV head), its keys and values — after an
// optional eviction gather (KV-Kaizen §3, long context: the evictor runs on the
// same cache and the ratios multiply) — quantised by the table's scheme
// (App. C.3: grouped asymmetric KIVI32, or the paper's symmetric per-row SYMROW),
// or as bf16 at b = 16 (§2.2: a b = 16 GQA layer is the uncompressed cache).
// The layout written is the one documented in include/kvk.h.
//
// One workgroup of 256 threads writes one 32-token block of one stream: it stages
// the block's K and V in LDS as fp32, computes the group metadata, then every
// thread assembles whole 32-bit words of codes so that the global stores are
// coalesced.
#include <hip/hip_runtime.h>

#include "kvk_device.h"
#include "kvk_internal.h"

using namespace kvkd;

namespace {

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
  int32_t kivi;
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

template <int D>
__global__ __launch_bounds__(256) void compress_kernel(CompressArgs a) {
  constexpr int LD = D + 1;  // padded LDS row
  __shared__ float Ks[32 * LD];
  __shared__ float Vs[32 * LD];
  __shared__ float kmeta[2 * D];          // KIVI: scale, zero per channel; SYMROW: row scale
  __shared__ float vmeta[2 * 32 * (D / 32)];

  const int tid = threadIdx.x;
  const int nblk = a.nbf + 1;
  const int stream = blockIdx.x / nblk;
  const int blk = blockIdx.x % nblk;
  const bool tail = blk == a.nbf;
  const int tok0 = blk * 32;
  const int ntok = tail ? a.n_stored - tok0 : 32;  // valid tokens of this block

  // ---- stage K and V (fp32) ----
  for (int idx = tid; idx < 32 * D; idx += 256) {
    const int t = idx / D, c = idx % D;
    float kv = 0.0f, vv = 0.0f;
    if (t < ntok) {
      int pos = tok0 + t;
      if (a.keep) {
        pos = a.keep[(int64_t)stream * a.n_stored + pos];
        pos = pos < 0 ? 0 : (pos >= a.n_tokens ? a.n_tokens - 1 : pos);
      }
      const int64_t e = ((int64_t)stream * a.n_tokens + pos) * D + c;
      if (a.in_f32) {
        kv = static_cast<const float*>(a.k)[e];
        vv = static_cast<const float*>(a.v)[e];
      } else {
        kv = bf16_to_f32(static_cast<const uint16_t*>(a.k)[e]);
        vv = bf16_to_f32(static_cast<const uint16_t*>(a.v)[e]);
      }
    }
    Ks[t * LD + c] = kv;
    Vs[t * LD + c] = vv;
  }
  __syncthreads();

  uint8_t* out = a.region + (int64_t)stream * a.stream_bytes +
                 (tail ? (int64_t)a.nb_cap * a.block_bytes : (int64_t)blk * a.block_bytes);

  if (tail || a.bits == 16) {
    // bf16 block: 16-byte chunks of 8 values, see the bf16 block layout.
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
          w[p] = (uint32_t)f32_to_bf16_bits(Vs[t0 * LD + c]) |
                 ((uint32_t)f32_to_bf16_bits(Vs[t1 * LD + c]) << 16);
        }
      }
      o4[ci] = make_uint4(w[0], w[1], w[2], w[3]);
    }
    return;
  }

  const int bits = a.bits;
  const float levels = (float)((1 << bits) - 1);

  // ---- group metadata ----
  if (a.kivi) {
    if (tid < D) {  // K: channel tid over the block's 32 tokens
      float mn = Ks[tid], mx = Ks[tid];
      for (int t = 1; t < 32; ++t) {
        const float x = Ks[t * LD + tid];
        mn = fminf(mn, x);
        mx = fmaxf(mx, x);
      }
      const _Float16 sh = (_Float16)((mx - mn) / levels);
      const _Float16 zh = (_Float16)mn;
      kmeta[tid] = (float)sh;
      kmeta[D + tid] = (float)zh;
    } else if (tid < 2 * D) {  // V: token t, channel group g
      const int r = tid - D, t = r / (D / 32), g = r % (D / 32);
      const float* row = &Vs[t * LD + 32 * g];
      float mn = row[0], mx = row[0];
      for (int c = 1; c < 32; ++c) {
        mn = fminf(mn, row[c]);
        mx = fmaxf(mx, row[c]);
      }
      const _Float16 sh = (_Float16)((mx - mn) / levels);
      const _Float16 zh = (_Float16)mn;
      vmeta[2 * (t * (D / 32) + g)] = (float)sh;
      vmeta[2 * (t * (D / 32) + g) + 1] = (float)zh;
    }
  } else if (tid < 64) {  // SYMROW: one scale per token row, K (tid < 32) and V
    const float* row = tid < 32 ? &Ks[tid * LD] : &Vs[(tid - 32) * LD];
    float amax = 0.0f;
    for (int c = 0; c < D; ++c) amax = fmaxf(amax, fabsf(row[c]));
    const float q = (float)((1 << (bits - 1)) - 1);
    const float sc = bf16_to_f32(f32_to_bf16_bits(amax / q));
    if (tid < 32) kmeta[tid] = sc;
    else vmeta[tid - 32] = sc;
  }
  __syncthreads();

  // ---- codes: whole 32-bit words ----
  uint32_t* ow = reinterpret_cast<uint32_t*>(out);
  const int cb = 4 * D * bits;          // bytes per code region
  const int lane_bytes_k = D * bits / 32;
  const int lane_bytes_v = D * bits / 16;
  for (int wi = tid; wi < 2 * cb / 4; wi += 256) {
    const bool isv = wi >= cb / 4;
    const int wb = 4 * (isv ? wi - cb / 4 : wi);  // byte offset inside the region
    int lam, r2, tau = 0;  // lane and byte of its share held by this word
    if (!isv) {
      tau = wb / (2 * D * bits);
      share_of(lane_bytes_k, wb % (2 * D * bits), lam, r2);
    } else {
      share_of(lane_bytes_v, wb, lam, r2);
    }
    const int i = lam & 15, kg = lam >> 4;
    // the slots held by this word: (chunk x, slot s, bit)
    int nslot, x0, s0;
    if (bits == 8) { nslot = 4; x0 = r2 / 8; s0 = 4 * ((r2 % 8) / 4); }
    else if (bits == 4) { nslot = 8; x0 = r2 / 4; s0 = 0; }
    else { nslot = 16; x0 = r2 / 2; s0 = 0; }
    uint32_t word = 0;
    for (int q = 0; q < nslot; ++q) {
      int x, s, bit;
      if (bits == 8) { x = x0; s = s0 + q; bit = 8 * q; }
      else if (bits == 4) { x = x0; s = q; bit = 16 * (s & 1) + 4 * (s >> 1); }
      else { x = x0 + (q >> 3); s = q & 7; bit = 16 * (s & 1) + 2 * (s >> 1) + 8 * (q >> 3); }
      uint32_t u;
      if (!isv) {
        const int t = 16 * tau + i, c = 32 * x + 8 * kg + s;
        const float xv = Ks[t * LD + c];
        u = a.kivi ? kivi_code(xv, kmeta[c], kmeta[D + c], levels) : sym_code(xv, kmeta[t], bits);
      } else {
        const int c = 16 * x + i, t = 16 * (s >> 2) + 4 * kg + (s & 3);
        const float xv = Vs[t * LD + c];
        if (a.kivi) {
          const int g = c >> 5;
          u = kivi_code(xv, vmeta[2 * (t * (D / 32) + g)], vmeta[2 * (t * (D / 32) + g) + 1], levels);
        } else {
          u = sym_code(xv, vmeta[t], bits);
        }
      }
      word |= u << bit;
    }
    ow[wi] = word;
  }

  // ---- metadata stores ----
  uint16_t* om = reinterpret_cast<uint16_t*>(out + 2 * cb);
  if (a.kivi) {
    for (int idx = tid; idx < 4 * D; idx += 256) {
      float val;
      if (idx < 2 * D) {
        val = kmeta[idx];  // scale[0..D) then zero[0..D)
      } else {
        const int e = idx - 2 * D;  // ((g*2 + w)*4 + kg)*8 + s
        const int s = e & 7, kg = (e >> 3) & 3, w = (e >> 5) & 1, g = e >> 6;
        const int t = 16 * (s >> 2) + 4 * kg + (s & 3);
        val = vmeta[2 * (t * (D / 32) + g) + w];
      }
      om[idx] = bitcast<uint16_t>((_Float16)val);  // exact: the value is an fp16
    }
  } else if (tid < 64) {
    om[tid] = f32_to_bf16_bits(tid < 32 ? kmeta[tid] : vmeta[tid - 32]);
  }
}

// Test-only dequantiser: one thread per (stream, token, channel).
template <int D>
__global__ __launch_bounds__(256) void dequant_kernel(const uint8_t* region, int64_t stream_bytes,
                                                      int64_t block_bytes, int nb_cap, int n_stored,
                                                      int n_streams, int bits, int kivi, float* kout,
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
    if (kivi) {
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
  if ((reinterpret_cast<uintptr_t>(arena) & 15) || (reinterpret_cast<uintptr_t>(k) & 3) ||
      (reinterpret_cast<uintptr_t>(v) & 3))
    return fail(KVK_ERR_INVALID, "misaligned buffer");
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
  a.kivi = d.qscheme == KVK_Q_KIVI32;
  const int64_t nstreams = (int64_t)d.batch * d.n_kv_heads;
  const int64_t grid = nstreams * (a.nbf + 1);
  if (grid > 0x7fffffffLL) return fail(KVK_ERR_UNSUPPORTED, "grid too large");
  if (d.head_dim == 128)
    hipLaunchKernelGGL(compress_kernel<128>, dim3((unsigned)grid), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(compress_kernel<64>, dim3((unsigned)grid), dim3(256), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(KVK_ERR_DEVICE, "compress launch: %s", hipGetErrorString(e));
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
  if (d.kind == KVK_MLA) return mla_debug_dequantize(t, layer, n_stored, arena, k_out, v_out, stream);
  const int a = t->info.anchor_of[layer];
  const uint8_t* region = static_cast<const uint8_t*>(arena) + t->info.layer_offset[a];
  const int nstreams = d.batch * d.n_kv_heads;
  const int64_t total = (int64_t)nstreams * n_stored * d.head_dim;
  const int64_t grid = (total + 255) / 256;
  if (grid > 0x7fffffffLL) return fail(KVK_ERR_UNSUPPORTED, "grid too large");
  const int kivi = d.qscheme == KVK_Q_KIVI32;
  if (d.head_dim == 128)
    hipLaunchKernelGGL(dequant_kernel<128>, dim3((unsigned)grid), dim3(256), 0, stream, region,
                       t->info.stream_bytes[a], t->block_bytes[a], t->nb_cap, n_stored, nstreams,
                       t->bits[a], kivi, k_out, v_out);
  else
    hipLaunchKernelGGL(dequant_kernel<64>, dim3((unsigned)grid), dim3(256), 0, stream, region,
                       t->info.stream_bytes[a], t->block_bytes[a], t->nb_cap, n_stored, nstreams,
                       t->bits[a], kivi, k_out, v_out);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(KVK_ERR_DEVICE, "dequantise launch: %s", hipGetErrorString(e));
  return KVK_OK;
}
