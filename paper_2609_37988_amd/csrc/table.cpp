// Host side of libkvk: plan validation, anchors, cost model, arena layout.
//
// Plans and actions follow §2.2 of KV-Kaizen (arXiv 2609.37988): eq. (1) gives
// each action's cost in bits per token, eq. (2) the plan's compression ratio
// against the bf16 GQA cache, eq. (3) the action set; §2.1 defines anchors (a
// layer owns a cache or inherits from the nearest anchor before it).  The
// storage accounting follows App. C.3.  Nothing in this file launches work on a
// device; it only asks the HIP runtime whether a buffer is GPU memory.
#include <cmath>
#include <cstdio>
#include <cstring>
#include <new>

#include "kvk_internal.h"

namespace kvk {

static thread_local std::string g_last_error;

void set_error(const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
}

kvk_status fail(kvk_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

kvk_status check_gpu_buffers(std::initializer_list<const void*> ptrs, const char* what) {
  int i = 0;
  for (const void* p : ptrs) {
    ++i;
    if (!p) continue;
    hipPointerAttribute_t a;
    const hipError_t e = hipPointerGetAttributes(&a, p);
    if (e != hipSuccess) (void)hipGetLastError();  // the query's error is not the caller's
    if (e != hipSuccess || a.type == hipMemoryTypeUnregistered)
      return fail(KVK_ERR_INVALID, "%s: buffer argument %d (%p) is not GPU-accessible memory", what, i, p);
  }
  return KVK_OK;
}

int64_t gqa_block_bytes(int32_t head_dim, int32_t bits, int32_t qscheme) {
  const int64_t D = head_dim;
  if (bits == 16) return 128 * D;                 // bf16 K and V, 32 tokens
  if (qscheme == KVK_Q_KIVI32) return 8 * D * (bits + 1);  // codes + fp16 (scale, zero)
  if (qscheme == KVK_Q_GROUP64) return 8 * D * bits + 4 * D;  // codes + fp16 (scale, zero) per 64 ch, K and V
  return 8 * D * bits + 128;                      // codes + bf16 row scales
}

int64_t gqa_split_target(const kvk_table* t, int32_t l0, int32_t l1) {
  // A wave pays its start (query, filling its prefetch ring) and its split
  // partial once, so splits are as long as the launch allows while it still has
  // about kSplitWaves waves: two rounds of the D1 wave slots of an MI355X (256 CUs
  // x 8 waves).  Measured on the 14B mixed stack: 1 MiB splits 3.54 ms, 2 MiB 3.44,
  // one split per stream (<= 4 MiB) 3.35.  Between 1 MiB and 16 MiB; computed from
  // the capacity, so the workspace size bounds every n_stored.  A per-sequence
  // table counts every sequence's distinct anchors.
  constexpr int64_t kSplitWaves = 4096;
  int64_t total = 0;
  const size_t n_seq = t->seq.empty() ? 1 : t->seq.size();
  for (size_t i = 0; i < n_seq; ++i) {
    const kvk_table* s = t->seq.empty() ? t : t->seq[i];
    bool seen[KVK_MAX_LAYERS] = {};
    for (int l = l0; l < l1; ++l) {
      const int32_t a = s->info.anchor_of[l];
      if (seen[a]) continue;
      seen[a] = true;
      total += (int64_t)s->d.batch * s->d.n_kv_heads * s->nb_cap * s->block_bytes[a];
    }
  }
  return total / kSplitWaves;  // clamped per precision by split_blocks_for
}

int32_t split_blocks_for(int32_t bits, int32_t qscheme, int32_t head_dim, int32_t n_blocks, int64_t target_bytes,
                         int32_t waves, int32_t* count_bound) {
  // target_bytes of cache per wave (gqa_split_target); the stream's blocks are
  // divided evenly so that no split is a short remainder, in a multiple of the
  // decode kernel's prefetch depth so that only a stream's last split runs past
  // its end.  A split read by `waves` chunk waves (an anchor with many reader rows)
  // is that many times as long: the launch's wave count is what the target sizes,
  // and every split re-reads the item's queries and writes partials for all its
  // rows (one anchor read by 48 layers at 14B: 240 rows, 61 KiB of queries and
  // 127 KiB of partials per split and stream; 357 MB of partials per step with
  // per-wave splits, 97 MB with 4x longer ones).
  const int64_t bb = gqa_block_bytes(head_dim, bits, qscheme);
  const int64_t nr = ring_depth_for(bits);
  // The 8- and 16-bit paths stream: splits between 1 and 16 MiB.  The 2- and 4-bit
  // paths are bound by their unpacking, not by the stream, so longer splits do not
  // pay there (14B eviction stack: 1 MiB 1.14 ms, 1.1 MiB 1.17 ms); their splits are
  // at most 1 MiB and shorter when the launch would otherwise hold fewer waves than
  // about two per wave slot (7B shape, 28 layers x 32 streams: 1 MiB splits gave the
  // int2 stack 896 waves for 2048 slots), down to 128 KiB.
  // The launch's bytes per wave (target_bytes) aim at about 4096 waves; per precision
  // that becomes about 512 for bf16 (streaming waves saturate HBM well before the
  // wave slots are full, and every split costs a start and a partial: the 7B-shaped
  // bf16 stack read whole streams, 896 waves, at 88 % of HBM against 81 % with 4
  // splits per stream), 2048 for the 2- and 4-bit items (one round of the wave slots:
  // the 7B int4 stack 62 % -> 64 %) and 4096 for int8 (3 splits per stream on the 7B
  // stack, 79 %, beat 1 and 2).  The 14B mixed and the 128k eviction stacks split as
  // before (their targets sit at the clamps).
  const int64_t w = waves > 1 ? waves : 1;
  const int64_t lo = w * (bits <= 4 ? (128LL << 10) : (1LL << 20)), hi = w * (bits <= 4 ? (1LL << 20) : (16LL << 20));
  target_bytes *= w * (bits == 16 ? 8 : (bits <= 4 ? 2 : 1));
  int64_t target = (target_bytes < lo ? lo : (target_bytes > hi ? hi : target_bytes)) / bb;
  if (target < nr) target = nr;
  const int64_t nb = n_blocks > 0 ? n_blocks : 1;
  int64_t nsplit = (nb + target - 1) / target;
  // The 2- and 4-bit items take one split fewer when the longer splits stay within
  // the clamp: the split count rounded down instead of up keeps a launch within one
  // round of the wave slots where rounding up spills into a second (the 7B int4 and
  // int2 stacks: 2 splits per stream, 1792 waves, 222 and 204 us, against 3 splits,
  // 2688 waves, 235 and 213 us).  The count stays at most the rounded-up count of
  // the capacity, so the workspace bound below still holds.
  if (bits <= 4 && nsplit > 1) {
    const int64_t nfloor = nb / target > 0 ? nb / target : 1;
    if (((nb + nfloor - 1) / nfloor + nr - 1) / nr * nr * bb <= hi) nsplit = nfloor;
  }
  int64_t per = (nb + nsplit - 1) / nsplit;
  per = (per + nr - 1) / nr * nr;
  // The split count ceil(nb / per) is at most nsplit, which grows with nb (the count
  // itself need not: rounding per up can save a split), so nsplit bounds the count of
  // every length up to n_blocks.
  if (count_bound) *count_bound = (int32_t)nsplit;
  return (int32_t)per;
}

int32_t gqa_item_split_blocks(const kvk_table* s, int32_t anchor, int32_t l0, int32_t l1, int32_t n_blocks,
                              int64_t target_bytes, int32_t* count_bound) {
  const int32_t G = s->d.n_q_heads / s->d.n_kv_heads;
  const int32_t rb = anchor > l0 ? anchor : l0;
  const int32_t re = s->next_anchor[anchor] < l1 ? s->next_anchor[anchor] : l1;
  const int32_t nch = (G * (re - rb) + 15) / 16;
  // Only the chunk waves of one workgroup (up to 4) lengthen the split: the several
  // workgroups of a larger unit drift apart over a long split and then read it from
  // HBM again (one int4 anchor for 48 layers at 14B, 16 chunk waves: FETCH 1.38x the
  // cache bytes with per-wave splits, 1.19x with 4x longer ones, 1.41x with 8x, 1.69x
  // with 16x).
  const int32_t w = gqa_chunk_waves(nch);
  return split_blocks_for(s->bits[anchor], s->d.qscheme, s->d.head_dim, n_blocks, target_bytes, w < 4 ? w : 4,
                          count_bound);
}

int64_t mla_block_bytes(int32_t W, int32_t bits, int32_t qscheme) {
  if (bits == 16) return 64LL * W;                          // bf16, 32 tokens
  if (qscheme == KVK_Q_KIVI32) return 4LL * W * (bits + 1);  // codes + fp16 (scale, zero) / 32 ch
  return 4LL * W * bits + 128;                              // codes + two bf16 scales / token
}

void mla_split_rule(const kvk_table* t, int32_t anchor, int32_t* target_out, int32_t* nr_out) {
  // A workgroup's time per block grows with the stored width W (scores over W
  // channels, the latent product over d) on top of a fixed part (softmax,
  // barriers): about W + 192 units.  Splits hold about 73728 units (96 blocks at
  // W = 576, 230 at W = 128), so that the workgroups of all widths take about the
  // same time and a step launches enough of them to balance the GPU; the split
  // partial (Hq * (d + 2) * 4 bytes) stays a few percent of a bf16 split.
#ifndef KVK_MLA_SPLIT_UNITS
#define KVK_MLA_SPLIT_UNITS 73728
#endif
  const int32_t W = t->rank[anchor] + t->d.rope_dim;
  const int64_t nr = (int64_t)mla_ring_depth(W, t->bits[anchor], t->d.qscheme == KVK_Q_KIVI32) *
                     mla_iter_blocks(W);  // blocks per pass of the ring
  // bf16 streams are bound by HBM and take twice as long splits (fewer workgroup
  // starts: MLA stack 0.96 -> 0.93 ms); the dequantising paths keep the shorter ones.
  // A bf16 anchor read by several layers (one workgroup per reader, sharing the
  // stream through L2) takes half the dequantising length instead: over longer
  // splits the readers drift apart and fetch the stream again (depth-grouped MLA
  // stack: 1.37x the cache bytes fetched at the long length, 1.19x at a quarter of
  // it, 705 -> 692 us; the int4 form is unchanged by the length, 1.16-1.17x, the
  // readers' absorbed queries).
  const bool shared = t->next_anchor[anchor] - anchor > 1;
  int64_t target = (int64_t)KVK_MLA_SPLIT_UNITS / (W + 192);
  if (t->bits[anchor] == 16) target = shared ? target / 2 : 2 * target;
  if (target < nr) target = nr;
  *target_out = (int32_t)target;
  *nr_out = (int32_t)nr;
}

int32_t mla_split_blocks_for(const kvk_table* t, int32_t anchor, int32_t n_blocks) {
  int32_t target = 0, nr = 1;
  mla_split_rule(t, anchor, &target, &nr);
  return mla_split_len(target, nr, n_blocks);
}

uint64_t fnv1a64(const uint8_t* p, size_t n) {
  uint64_t h = 0xcbf29ce484222325ull;
  for (size_t i = 0; i < n; ++i) h = (h ^ p[i]) * 0x100000001b3ull;
  return h;
}

int32_t mla_units(const kvk_table* t, int32_t anchor, int32_t n_stored) {
  const int32_t nb = n_stored / KVK_GROUP;
  const int32_t u = n_splits(nb, mla_split_blocks_for(t, anchor, nb));
  return u > 0 ? u : 1;
}

void mla_workspace(const kvk_table* t, int32_t l0, int32_t l1, MlaWorkspace* ws) {
  const kvk_dims& d = t->d;
  int64_t off = 0;
  for (int l = l0; l < l1; ++l) {
    const int32_t a = t->info.anchor_of[l];
    ws->q_off[l] = off;
    off += round256((int64_t)d.batch * mla_heads_padded(d.n_q_heads) * (t->rank[a] + d.rope_dim) * 2);
  }
  for (int l = l0; l < l1; ++l) {
    const int32_t a = t->info.anchor_of[l];
    int32_t target = 0, nr = 1;
    mla_split_rule(t, a, &target, &nr);
    ws->units_cap[l] = mla_units_bound(target, t->nb_cap);  // every n_stored <= cap
    ws->part_off[l] = off;
    off += round256((int64_t)d.batch * ws->units_cap[l] * mla_heads_padded(d.n_q_heads) * (t->rank[a] + 2) * 4);
  }
  ws->total = off;
}

}  // namespace kvk

using namespace kvk;

static kvk_status validate_mla(const kvk_dims& d, const kvk_action* plan) {
  if (d.n_q_heads < 8 || d.n_q_heads % 8 != 0 || d.n_q_heads > 256)
    return fail(KVK_ERR_UNSUPPORTED, "MLA n_q_heads %d must be a multiple of 8 up to 256",
                d.n_q_heads);
  if (d.n_kv_heads < 1 || d.head_dim < 1)
    return fail(KVK_ERR_INVALID, "MLA n_kv_heads/head_dim (the bf16 GQA reference of eq. (2)) must be >= 1");
  if (d.latent_dim < 256 || d.latent_dim % 256 != 0)
    return fail(KVK_ERR_INVALID,
                "latent_dim %d must be a positive multiple of 256 (every rank in {r/8..r} a multiple of 32)",
                d.latent_dim);
  if (d.rope_dim != 64) return fail(KVK_ERR_UNSUPPORTED, "rope_dim %d: only 64 is provided", d.rope_dim);
  if (d.nope_dim < 32 || d.nope_dim % 32 != 0 || d.nope_dim > 256)
    return fail(KVK_ERR_UNSUPPORTED, "nope_dim %d must be a multiple of 32 up to 256", d.nope_dim);
  if (d.v_dim < 16 || d.v_dim % 16 != 0 || d.v_dim > 256)
    return fail(KVK_ERR_UNSUPPORTED, "v_dim %d must be a multiple of 16 up to 256", d.v_dim);
  const int32_t r = d.latent_dim;
  for (int l = 0; l < d.n_layers; ++l) {
    const kvk_action& a = plan[l];
    if (a.inherit) continue;
    if (a.rank != r && a.rank != r / 2 && a.rank != r / 4 && a.rank != r / 8)
      return fail(KVK_ERR_INVALID, "layer %d: rank %d not in {r/8, r/4, r/2, r} with r = %d", l,
                  a.rank, r);
    if (a.rank > 1024)
      return fail(KVK_ERR_UNSUPPORTED, "layer %d: kept width %d above 1024 is not provided", l, a.rank);
  }
  return KVK_OK;
}

static bool is_bits(int32_t b) { return b == 2 || b == 4 || b == 8 || b == 16; }

extern "C" kvk_status kvk_layer_table(const kvk_dims* dims, const kvk_action* plan,
                                      kvk_table** out) {
  if (!dims || !plan || !out) return fail(KVK_ERR_INVALID, "kvk_layer_table: NULL argument");
  *out = nullptr;
  const kvk_dims& d = *dims;
  if (d.kind != KVK_GQA && d.kind != KVK_MLA)
    return fail(KVK_ERR_INVALID, "kind %d is neither GQA nor MLA", d.kind);
  const bool mla = d.kind == KVK_MLA;
  if (d.n_layers < 1 || d.n_layers > KVK_MAX_LAYERS)
    return fail(KVK_ERR_INVALID, "n_layers %d outside 1..%d", d.n_layers, KVK_MAX_LAYERS);
  if (!mla) {
    if (d.n_kv_heads < 1 || d.n_q_heads < 1 || d.n_q_heads % d.n_kv_heads != 0)
      return fail(KVK_ERR_INVALID, "n_q_heads %d must be a positive multiple of n_kv_heads %d",
                  d.n_q_heads, d.n_kv_heads);
    if (d.head_dim != 64 && d.head_dim != 128)
      return fail(KVK_ERR_UNSUPPORTED, "head_dim %d not in {64, 128}", d.head_dim);
  }
  if (d.qscheme != KVK_Q_KIVI32 && d.qscheme != KVK_Q_SYMROW && d.qscheme != KVK_Q_GROUP64)
    return fail(KVK_ERR_INVALID, "qscheme %d unknown", d.qscheme);
  if (d.qscheme == KVK_Q_GROUP64 && d.kind != KVK_GQA)
    return fail(KVK_ERR_UNSUPPORTED, "GROUP64 is built for GQA tables only");
  if (d.batch < 1 || d.max_tokens < 1)
    return fail(KVK_ERR_INVALID, "batch %d and max_tokens %d must be >= 1", d.batch, d.max_tokens);
  if (d.keep_tokens < 0 || d.keep_tokens > d.max_tokens)
    return fail(KVK_ERR_INVALID, "keep_tokens %d outside 0..max_tokens", d.keep_tokens);
  if (plan[0].inherit)
    return fail(KVK_ERR_INVALID, "layer 0 must own a cache (it has no earlier anchor)");
  const int32_t width = 2 * d.n_kv_heads * d.head_dim;  // cached scalars per token, bf16 GQA
  for (int l = 0; l < d.n_layers; ++l) {
    const kvk_action& a = plan[l];
    if (a.inherit) continue;
    if (!is_bits(a.bits)) return fail(KVK_ERR_INVALID, "layer %d: bits %d not in {2,4,8,16}", l, a.bits);
    if (!mla && a.rank != 0 && a.rank != width)
      return fail(KVK_ERR_INVALID, "layer %d: GQA has no rank axis (rank %d)", l, a.rank);
  }
  if (mla) {
    const kvk_status st = validate_mla(d, plan);
    if (st != KVK_OK) return st;
  }
  // The decode kernels address a stream through a 32-bit byte range (buffer
  // resources and work-item fields), so every stream stays below 2 GiB.
  {
    const int64_t cap = d.keep_tokens > 0 ? d.keep_tokens : d.max_tokens;
    for (int l = 0; l < d.n_layers; ++l) {
      const kvk_action& a = plan[l];
      if (a.inherit) continue;
      const int32_t per_tok = mla ? a.rank + d.rope_dim : 2 * d.head_dim;
      const int64_t bb = mla ? mla_block_bytes(per_tok, a.bits, d.qscheme) : gqa_block_bytes(d.head_dim, a.bits, d.qscheme);
      const int64_t sb = round256(cap / KVK_GROUP * bb + 64LL * per_tok);
      if (sb > 0x7fffffffLL)
        return fail(KVK_ERR_UNSUPPORTED, "layer %d: a stream of %lld bytes at %lld stored tokens; streams are limited to 2 GiB",
                    l, (long long)sb, (long long)cap);
    }
  }
  const int64_t streams = mla ? (int64_t)d.batch : (int64_t)d.batch * d.n_kv_heads;

  kvk_table* t = new (std::nothrow) kvk_table();
  if (!t) return fail(KVK_ERR_INVALID, "out of host memory");
  t->d = d;
  std::memcpy(t->plan, plan, sizeof(kvk_action) * d.n_layers);
  t->cap = d.keep_tokens > 0 ? d.keep_tokens : d.max_tokens;
  t->nb_cap = t->cap / KVK_GROUP;

  kvk_table_info& inf = t->info;
  std::memset(&inf, 0, sizeof(inf));
  inf.stored_tokens_cap = t->cap;
  inf.c0_bits_per_token = (double)d.n_layers * width * 16.0;  // eq. (2)
  int64_t offset = 0;
  int32_t last = -1;
  double total_cost = 0.0;
  int64_t stored_alg = 0;
  for (int l = 0; l < d.n_layers; ++l) {
    const kvk_action& a = plan[l];
    inf.layer_offset[l] = -1;
    if (!a.inherit) {
      last = l;
      t->bits[l] = a.bits;
      // Scalars one stream stores per token: GQA K and V of one head; MLA c[:d] and k^R.
      const int32_t per_tok = mla ? a.rank + d.rope_dim : 2 * d.head_dim;
      t->rank[l] = mla ? a.rank : 0;
      t->block_bytes[l] = mla ? mla_block_bytes(per_tok, a.bits, d.qscheme)
                              : gqa_block_bytes(d.head_dim, a.bits, d.qscheme);
      const int64_t sb = round256(t->nb_cap * t->block_bytes[l] + 64LL * per_tok);
      inf.stream_bytes[l] = sb;
      inf.layer_bytes[l] = sb * streams;
      inf.layer_offset[l] = offset;
      offset += round256(inf.layer_bytes[l]);
      // eq. (1): (d + d_R) b; for GQA d = 2 n_kv d_h and d_R = 0.
      inf.layer_cost_bits[l] = mla ? (double)per_tok * a.bits : (double)width * a.bits;
      const int64_t per_stream = (int64_t)t->nb_cap * t->block_bytes[l] +
                                 (int64_t)(t->cap % KVK_GROUP) * 2 * per_tok;
      inf.layer_bits_per_elt[l] = t->cap ? per_stream * 8.0 / ((double)t->cap * per_tok) : 0.0;
      stored_alg += per_stream * streams;
      inf.n_anchors++;
    } else {
      t->bits[l] = 0;
      t->rank[l] = 0;
      inf.layer_cost_bits[l] = 0.0;
    }
    inf.anchor_of[l] = last;
    total_cost += inf.layer_cost_bits[l];
  }
  for (int l = d.n_layers - 1, nxt = d.n_layers; l >= 0; --l) {
    t->next_anchor[l] = nxt;
    if (!plan[l].inherit) nxt = l;
  }
  inf.arena_bytes = offset;
  inf.cost_bits_per_token = total_cost;
  inf.rho = inf.c0_bits_per_token / total_cost;
  const double bf16_full = (double)d.n_layers * d.batch * d.max_tokens * width * 2.0;
  inf.rho_realized = stored_alg > 0 ? bf16_full / (double)stored_alg : 0.0;
  size_t ws = 0;
  kvk_status st = kvk_workspace_bytes(t, 0, d.n_layers, &ws);
  if (st != KVK_OK) {
    delete t;
    return st;
  }
  inf.workspace_bytes = (int64_t)ws;
  *out = t;
  return KVK_OK;
}

extern "C" kvk_status kvk_table_query(const kvk_table* t, kvk_table_info* out) {
  if (!t || !out) return fail(KVK_ERR_INVALID, "kvk_table_query: NULL argument");
  *out = t->info;
  return KVK_OK;
}

extern "C" void kvk_table_destroy(kvk_table* t) { delete t; }

extern "C" kvk_status kvk_layer_table_batched(const kvk_dims* dims, const kvk_action* plans,
                                              kvk_table** out) {
  if (!dims || !plans || !out) return fail(KVK_ERR_INVALID, "kvk_layer_table_batched: NULL argument");
  *out = nullptr;
  const kvk_dims& d = *dims;
  if (d.batch < 1 || d.batch > KVK_MAX_BATCH_PLANS)
    return fail(KVK_ERR_INVALID, "batch %d outside 1..%d for per-sequence plans", d.batch, KVK_MAX_BATCH_PLANS);
  if (d.n_layers < 1 || d.n_layers > KVK_MAX_LAYERS)
    return fail(KVK_ERR_INVALID, "n_layers %d outside 1..%d", d.n_layers, KVK_MAX_LAYERS);
  kvk_table* t = new (std::nothrow) kvk_table();
  if (!t) return fail(KVK_ERR_INVALID, "out of host memory");
  kvk_dims one = d;
  one.batch = 1;
  int64_t base = 0;
  double cost = 0.0, stored = 0.0;
  for (int b = 0; b < d.batch; ++b) {
    kvk_table* s = nullptr;
    const kvk_status st = kvk_layer_table(&one, plans + (int64_t)b * d.n_layers, &s);
    if (st != KVK_OK) {
      delete t;
      return st;
    }
    t->seq.push_back(s);
    t->seq_base.push_back(base);
    base += round256(s->info.arena_bytes);
    cost += s->info.cost_bits_per_token;
    stored += s->info.rho_realized > 0 ? (double)d.n_layers * d.max_tokens * 4.0 * d.n_kv_heads * d.head_dim /
                                             s->info.rho_realized
                                       : 0.0;
  }
  t->d = d;
  t->cap = t->seq[0]->cap;
  t->nb_cap = t->seq[0]->nb_cap;
  kvk_table_info& inf = t->info;
  std::memset(&inf, 0, sizeof(inf));
  for (int l = 0; l < d.n_layers; ++l) {
    inf.anchor_of[l] = -1;
    inf.layer_offset[l] = -1;
  }
  inf.arena_bytes = base;
  inf.stored_tokens_cap = t->cap;
  inf.c0_bits_per_token = t->seq[0]->info.c0_bits_per_token;
  inf.cost_bits_per_token = cost / d.batch;  // the batch's mean plan
  inf.rho = inf.c0_bits_per_token / inf.cost_bits_per_token;
  const double bf16_full = (double)d.n_layers * d.batch * d.max_tokens * 4.0 * d.n_kv_heads * d.head_dim;
  inf.rho_realized = stored > 0 ? bf16_full / stored : 0.0;
  for (const kvk_table* s : t->seq) inf.n_anchors += s->info.n_anchors;
  size_t ws = 0;
  const kvk_status st = kvk_workspace_bytes(t, 0, d.n_layers, &ws);
  if (st != KVK_OK) {
    delete t;
    return st;
  }
  inf.workspace_bytes = (int64_t)ws;
  *out = t;
  return KVK_OK;
}

extern "C" kvk_status kvk_table_sequence_query(const kvk_table* t, int32_t b, kvk_table_info* out) {
  if (!t || !out) return fail(KVK_ERR_INVALID, "kvk_table_sequence_query: NULL argument");
  if (t->seq.empty()) return fail(KVK_ERR_INVALID, "not a table with per-sequence plans");
  if (b < 0 || b >= (int32_t)t->seq.size()) return fail(KVK_ERR_INVALID, "sequence %d out of range", b);
  *out = t->seq[b]->info;
  for (int l = 0; l < t->d.n_layers; ++l)
    if (out->layer_offset[l] >= 0) out->layer_offset[l] += t->seq_base[b];
  return KVK_OK;
}

extern "C" kvk_status kvk_workspace_bytes(const kvk_table* t, int32_t l0, int32_t l1, size_t* out) {
  if (!t || !out) return fail(KVK_ERR_INVALID, "kvk_workspace_bytes: NULL argument");
  if (l0 < 0 || l1 > t->d.n_layers || l0 >= l1)
    return fail(KVK_ERR_INVALID, "layer range [%d, %d) invalid for %d layers", l0, l1, t->d.n_layers);
  const kvk_dims& d = t->d;
  if (d.kind == KVK_MLA && t->seq.empty()) {
    MlaWorkspace ws;
    mla_workspace(t, l0, l1, &ws);
    *out = (size_t)ws.total;
    return KVK_OK;
  }
  if (!t->seq.empty()) {
    // The device-side work list, then GQA: every sequence's split partials (each
    // sized with its own, smaller, split target: the batch's longer splits need no
    // more); MLA: every sequence's own workspace, one after the other.
    size_t total;
    if (d.kind == KVK_MLA) {
      MlaSeqList L;
      if (kvk_status st = mla_seq_list(t, l0, l1, L, false)) return st;
      total = (size_t)L.bytes;
    } else {
      total = (size_t)gqa_batched_list_bytes(t, l0, l1);
    }
    for (const kvk_table* s : t->seq) {
      size_t one = 0;
      const kvk_status st = kvk_workspace_bytes(s, l0, l1, &one);
      if (st != KVK_OK) return st;
      total += one;
    }
    *out = total;
    return KVK_OK;
  }
  const int32_t G = d.n_q_heads / d.n_kv_heads;
  // Split partials: per query row (layer, b, head) and split, (o[d_h], m, l, 2 pad) in fp32.
  const int32_t nblk = t->nb_cap;  // full blocks; the tail is merged by the combine kernel
  const int64_t target = gqa_split_target(t, l0, l1);
  size_t floats = 0;
  for (int l = l0; l < l1; ++l) {
    const int32_t a = t->info.anchor_of[l];
    int32_t bound = 0;  // the splits of every n_stored up to the capacity
    gqa_item_split_blocks(t, a, l0, l1, nblk, target, &bound);
    floats += (size_t)d.batch * d.n_kv_heads * G * bound * (d.head_dim + 4);
  }
  *out = (size_t)round256((int64_t)(floats * sizeof(float)));
  return KVK_OK;
}

extern "C" kvk_status kvk_set_mla_weights(kvk_table* t, const void* w_uk, const void* w_uv) {
  if (!t) return fail(KVK_ERR_INVALID, "kvk_set_mla_weights: NULL table");
  if (t->d.kind != KVK_MLA) return fail(KVK_ERR_INVALID, "kvk_set_mla_weights: an MLA table is required");
  if (!w_uk != !w_uv) return fail(KVK_ERR_INVALID, "kvk_set_mla_weights: pass both weights or neither");
  if ((reinterpret_cast<uintptr_t>(w_uk) & 15) || (reinterpret_cast<uintptr_t>(w_uv) & 15))
    return fail(KVK_ERR_INVALID, "kvk_set_mla_weights: misaligned weights (16 bytes required)");
  if (w_uk)
    if (kvk_status st = check_gpu_buffers({w_uk, w_uv}, "kvk_set_mla_weights")) return st;
  t->mla_w_uk = w_uk;
  t->mla_w_uv = w_uv;
  return KVK_OK;
}

extern "C" double kvk_realized_bits(int32_t qscheme, int32_t bits, int32_t group, int64_t window,
                                    int64_t context) {
  if (!is_bits(bits) || context <= 0 || window < 0 || window > context) return -1.0;
  double per;
  if (qscheme == KVK_Q_SYMROW) {
    per = bits + 16.0 / 128.0;  // one bf16 scale per 128-element token-head row
  } else if (qscheme == KVK_Q_KIVI32 || qscheme == KVK_Q_GROUP64) {
    if (group <= 0) return -1.0;
    per = bits + 32.0 / group;  // fp16 scale + fp16 zero per group
  } else {
    return -1.0;
  }
  return (per * (double)(context - window) + 16.0 * (double)window) / (double)context;
}

extern "C" kvk_status kvk_rho_range(int32_t n_layers, int32_t kv_width, int32_t latent_dim,
                                    int32_t rope_dim, int32_t mla, int32_t axes, double* rho_min,
                                    double* rho_max) {
  if (!rho_min || !rho_max || n_layers < 1 || kv_width < 1 || (mla && latent_dim < 8))
    return fail(KVK_ERR_INVALID, "kvk_rho_range: invalid arguments");
  const bool prec = axes & 1, rank = axes & 2, depth = axes & 4;
  const int nb = prec ? 4 : 1;
  const int32_t bset[4] = {16, 8, 4, 2};
  double cmin = 1e300, cmax = 0.0;
  for (int i = 0; i < nb; ++i) {
    const int32_t b = bset[i];
    const int nd = (mla && rank) ? 4 : 1;
    for (int k = 0; k < nd; ++k) {
      const double c = mla ? (double)(latent_dim / (1 << k) + rope_dim) * b : (double)kv_width * b;
      if (c < cmin) cmin = c;
      if (c > cmax) cmax = c;
    }
  }
  const double c0 = (double)n_layers * kv_width * 16.0;  // eq. (2)
  *rho_min = c0 / (n_layers * cmax);                     // eq. (5)
  *rho_max = depth ? c0 / cmin : c0 / (n_layers * cmin);
  return KVK_OK;
}

extern "C" const char* kvk_last_error(void) { return kvk::g_last_error.c_str(); }

extern "C" const char* kvk_version(void) { return "kvk 0.1 (gfx950)"; }
