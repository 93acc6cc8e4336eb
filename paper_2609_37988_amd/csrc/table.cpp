// Host side of libkvk: plan validation, anchors, cost model, arena layout.
//
// Plans and actions follow §2.2 of KV-Kaizen (arXiv 2609.37988): eq. (1) gives
// each action's cost in bits per token, eq. (2) the plan's compression ratio
// against the bf16 GQA cache, eq. (3) the action set; §2.1 defines anchors (a
// layer owns a cache or inherits from the nearest anchor before it).  The
// storage accounting follows App. C.3.  Nothing in this file touches a device.
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

int64_t gqa_block_bytes(int32_t head_dim, int32_t bits, int32_t qscheme) {
  const int64_t D = head_dim;
  if (bits == 16) return 128 * D;                 // bf16 K and V, 32 tokens
  if (qscheme == KVK_Q_KIVI32) return 8 * D * (bits + 1);  // codes + fp16 (scale, zero)
  return 8 * D * bits + 128;                      // codes + bf16 row scales
}

int32_t ring_depth_for(int32_t bits) {
  return bits == 16 ? 2 : (bits == 8 ? 2 : (bits == 4 ? 4 : 6));
}

int32_t split_blocks_for(int32_t bits, int32_t qscheme, int32_t head_dim, int32_t n_blocks) {
  // About 1 MiB of cache per wave: a wave pays one memory latency to start, so
  // longer splits amortise it (and the split partial); the stream's blocks are
  // divided evenly so that no split is a short remainder, in a multiple of the
  // decode kernel's prefetch depth so that only a stream's last split runs past
  // its end.
#ifndef KVK_SPLIT_TARGET
#define KVK_SPLIT_TARGET (1024 * 1024)
#endif
  const int64_t bb = gqa_block_bytes(head_dim, bits, qscheme);
  const int64_t nr = ring_depth_for(bits);
  int64_t target = KVK_SPLIT_TARGET / bb;
  if (target < nr) target = nr;
  const int64_t nb = n_blocks > 0 ? n_blocks : 1;
  const int64_t nsplit = (nb + target - 1) / target;
  int64_t per = (nb + nsplit - 1) / nsplit;
  per = (per + nr - 1) / nr * nr;
  return (int32_t)per;
}

}  // namespace kvk

using namespace kvk;

static bool is_bits(int32_t b) { return b == 2 || b == 4 || b == 8 || b == 16; }

extern "C" kvk_status kvk_layer_table(const kvk_dims* dims, const kvk_action* plan,
                                      kvk_table** out) {
  if (!dims || !plan || !out) return fail(KVK_ERR_INVALID, "kvk_layer_table: NULL argument");
  *out = nullptr;
  const kvk_dims& d = *dims;
  if (d.kind != KVK_GQA && d.kind != KVK_MLA)
    return fail(KVK_ERR_INVALID, "kind %d is neither GQA nor MLA", d.kind);
  if (d.kind == KVK_MLA)
    return fail(KVK_ERR_UNSUPPORTED, "MLA latent caches are not provided by this build");
  if (d.n_layers < 1 || d.n_layers > KVK_MAX_LAYERS)
    return fail(KVK_ERR_INVALID, "n_layers %d outside 1..%d", d.n_layers, KVK_MAX_LAYERS);
  if (d.n_kv_heads < 1 || d.n_q_heads < 1 || d.n_q_heads % d.n_kv_heads != 0)
    return fail(KVK_ERR_INVALID, "n_q_heads %d must be a positive multiple of n_kv_heads %d",
                d.n_q_heads, d.n_kv_heads);
  if (d.head_dim != 64 && d.head_dim != 128)
    return fail(KVK_ERR_UNSUPPORTED, "head_dim %d not in {64, 128}", d.head_dim);
  if (d.qscheme != KVK_Q_KIVI32 && d.qscheme != KVK_Q_SYMROW)
    return fail(KVK_ERR_INVALID, "qscheme %d unknown", d.qscheme);
  if (d.batch < 1 || d.max_tokens < 1)
    return fail(KVK_ERR_INVALID, "batch %d and max_tokens %d must be >= 1", d.batch, d.max_tokens);
  if (d.keep_tokens < 0 || d.keep_tokens > d.max_tokens)
    return fail(KVK_ERR_INVALID, "keep_tokens %d outside 0..max_tokens", d.keep_tokens);
  const int32_t G = d.n_q_heads / d.n_kv_heads;
  if (plan[0].inherit)
    return fail(KVK_ERR_INVALID, "layer 0 must own a cache (it has no earlier anchor)");
  const int32_t width = 2 * d.n_kv_heads * d.head_dim;
  for (int l = 0; l < d.n_layers; ++l) {
    const kvk_action& a = plan[l];
    if (a.inherit) continue;
    if (!is_bits(a.bits)) return fail(KVK_ERR_INVALID, "layer %d: bits %d not in {2,4,8,16}", l, a.bits);
    if (a.rank != 0 && a.rank != width)
      return fail(KVK_ERR_INVALID, "layer %d: GQA has no rank axis (rank %d)", l, a.rank);
  }

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
  int32_t max_readers = 0, run = 0;
  double total_cost = 0.0;
  int64_t stored_alg = 0;
  for (int l = 0; l < d.n_layers; ++l) {
    const kvk_action& a = plan[l];
    inf.layer_offset[l] = -1;
    if (!a.inherit) {
      last = l;
      run = 0;
      t->bits[l] = a.bits;
      t->block_bytes[l] = gqa_block_bytes(d.head_dim, a.bits, d.qscheme);
      const int64_t sb = round256(t->nb_cap * t->block_bytes[l] + 128LL * d.head_dim);
      inf.stream_bytes[l] = sb;
      inf.layer_bytes[l] = sb * d.batch * d.n_kv_heads;
      inf.layer_offset[l] = offset;
      offset += round256(inf.layer_bytes[l]);
      inf.layer_cost_bits[l] = (double)width * a.bits;  // eq. (1) with d = 2 n_kv d_h, d_R = 0
      const int64_t per_stream = (int64_t)t->nb_cap * t->block_bytes[l] +
                                 (int64_t)(t->cap % KVK_GROUP) * 4 * d.head_dim;
      inf.layer_bits_per_elt[l] = t->cap ? per_stream * 8.0 / ((double)t->cap * 2 * d.head_dim) : 0.0;
      stored_alg += per_stream * d.batch * d.n_kv_heads;
      inf.n_anchors++;
    } else {
      t->bits[l] = 0;
      inf.layer_cost_bits[l] = 0.0;
    }
    ++run;
    if (run > max_readers) max_readers = run;
    inf.anchor_of[l] = last;
    total_cost += inf.layer_cost_bits[l];
  }
  for (int l = d.n_layers - 1, nxt = d.n_layers; l >= 0; --l) {
    t->next_anchor[l] = nxt;
    if (!plan[l].inherit) nxt = l;
  }
  if ((int64_t)G * max_readers > 64) {
    delete t;
    return fail(KVK_ERR_UNSUPPORTED,
                "an anchor serves %d layers x %d query heads per KV head = %d > 64 query rows",
                max_readers, G, max_readers * G);
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

extern "C" kvk_status kvk_workspace_bytes(const kvk_table* t, int32_t l0, int32_t l1, size_t* out) {
  if (!t || !out) return fail(KVK_ERR_INVALID, "kvk_workspace_bytes: NULL argument");
  if (l0 < 0 || l1 > t->d.n_layers || l0 >= l1)
    return fail(KVK_ERR_INVALID, "layer range [%d, %d) invalid for %d layers", l0, l1, t->d.n_layers);
  const kvk_dims& d = t->d;
  const int32_t G = d.n_q_heads / d.n_kv_heads;
  // Split partials: per query row (layer, b, head) and split, (o[d_h], m, l, 2 pad) in fp32.
  const int32_t nblk = t->nb_cap;  // full blocks; the tail is merged by the combine kernel
  size_t floats = 0;
  for (int l = l0; l < l1; ++l) {
    const int32_t a = t->info.anchor_of[l];
    const int32_t sb = split_blocks_for(t->bits[a], d.qscheme, d.head_dim, nblk);
    floats += (size_t)d.batch * d.n_kv_heads * G * n_splits(nblk, sb) * (d.head_dim + 4);
  }
  *out = (size_t)round256((int64_t)(floats * sizeof(float)));
  return KVK_OK;
}

extern "C" double kvk_realized_bits(int32_t qscheme, int32_t bits, int32_t group, int64_t window,
                                    int64_t context) {
  if (!is_bits(bits) || context <= 0 || window < 0 || window > context) return -1.0;
  double per;
  if (qscheme == KVK_Q_SYMROW) {
    per = bits + 16.0 / 128.0;  // one bf16 scale per 128-element token-head row
  } else if (qscheme == KVK_Q_KIVI32) {
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
