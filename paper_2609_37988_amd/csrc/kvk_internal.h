// Internal declarations shared by the host-side translation units of libkvk.
#pragma once

#include <cstdarg>
#include <cstdint>
#include <initializer_list>
#include <mutex>
#include <string>
#include <vector>

#include "kvk.h"

struct kvk_table {
  kvk_dims d;
  kvk_action plan[KVK_MAX_LAYERS];
  kvk_table_info info;
  int32_t bits[KVK_MAX_LAYERS];         // bits of each layer's own action (anchors)
  int32_t rank[KVK_MAX_LAYERS];         // MLA: kept latent width d of each anchor
  int64_t block_bytes[KVK_MAX_LAYERS];  // bytes of one 32-token block (anchors)
  int32_t next_anchor[KVK_MAX_LAYERS];  // first anchor after l (n_layers if none)
  int32_t cap;                          // stored tokens capacity per stream
  int32_t nb_cap;                       // full-block capacity per stream (cap / 32)
  // Per-sequence plans: sequence b is the one-sequence table seq[b], whose arena sits
  // at byte seq_base[b] of the batch's arena.  Empty for a table with one plan.
  std::vector<kvk_table*> seq;
  std::vector<int64_t> seq_base;
  // Per-sequence plans: the workspaces kvk_decode_setup has written a decode work list
  // to (workspace address, layer range, hash of the list).  The only mutable part of a
  // table; guarded by setup_mu.
  struct DecodeSetup {
    const void* workspace;
    int32_t l0, l1;
    uint64_t hash;
    // MLA: the list's launch sizes, so that decode calls need not rebuild it
    int64_t rows_off = 0, items_off[4] = {0, 0, 0, 0};
    int32_t n_items[4] = {0, 0, 0, 0};
    int64_t n_wg[4] = {0, 0, 0, 0};
    int32_t dmax = 0;
  };
  mutable std::mutex setup_mu;
  mutable std::vector<DecodeSetup> setups;
  // MLA: the all-layer W_UK (latent-major) and W_UV attached by kvk_set_mla_weights
  // (caller-owned device memory), used by decode calls that pass no weights.
  const void* mla_w_uk = nullptr;
  const void* mla_w_uv = nullptr;
  ~kvk_table() {
    for (kvk_table* s : seq) delete s;
  }
};

namespace kvk {

// Thread-local last-error message.
void set_error(const char* fmt, ...);
kvk_status fail(kvk_status st, const char* fmt, ...);

inline int64_t round256(int64_t n) { return (n + 255) / 256 * 256; }

// Every buffer a kernel dereferences must be memory the HIP runtime maps for the GPU
// (a device allocation, or pinned or managed host memory): a pageable host pointer
// would fault the GPU.  Checked before any launch; NULL entries (optional buffers)
// are skipped.  `what` names the entry point in the error message.
kvk_status check_gpu_buffers(std::initializer_list<const void*> ptrs, const char* what);

// A list whose first N elements live inside the object (no heap allocation while
// it holds at most N: the one-plan decode path, bounded by the layer count) and
// which moves to the heap beyond that (per-sequence plans).  T trivially copyable.
template <class T, int N>
struct SmallVec {
  T local[N];
  std::vector<T> big;
  T* p = local;
  size_t n = 0;
  void resize(size_t m) {
    if (m > (size_t)N) {
      big.resize(m);
      p = big.data();
    }
    n = m;
  }
  void push_back(const T& v) {
    if (n < (size_t)N && big.empty()) {
      local[n++] = v;
      return;
    }
    if (big.empty()) big.assign(local, local + n);
    big.push_back(v);
    p = big.data();
    ++n;
  }
  T& operator[](size_t i) { return p[i]; }
  const T& operator[](size_t i) const { return p[i]; }
  size_t size() const { return n; }
};

// Bytes of one 32-token block of a GQA stream with `bits`-bit codes.
int64_t gqa_block_bytes(int32_t head_dim, int32_t bits, int32_t qscheme);

// Blocks the decode kernel keeps in flight per wave for a `bits`-bit anchor
// (must equal the kernel's ring depth).
// Blocks the GQA decode kernel keeps in flight per wave (registers), by bit-width:
// about 8-16 KiB of cache ahead of use within the register budget of two waves per
// SIMD.  Shared by the host (split lengths) and the kernel.
constexpr int gqa_ring_depth(int bits) { return bits == 16 ? 2 : (bits == 8 ? 2 : (bits == 4 ? 4 : 6)); }
inline int32_t ring_depth_for(int32_t bits) { return gqa_ring_depth(bits); }

// Blocks processed per split of the decode kernel for a `bits`-bit anchor whose
// streams hold n_blocks full blocks.  *count_bound (if given) receives a bound of the
// split count of every length up to n_blocks, so that a workspace sized with it at
// the capacity covers every n_stored (the count itself is not monotone in the
// length).  `waves` D1 waves read each split (an item's chunk waves), so its target
// and its bounds are that many times the per-wave ones.
int32_t split_blocks_for(int32_t bits, int32_t qscheme, int32_t head_dim, int32_t n_blocks, int64_t target_bytes,
                         int32_t waves, int32_t* count_bound = nullptr);
// D1 waves per (stream, split) of an item whose anchor's readers give nch 16-row
// query chunks: 1, 2, or a multiple of 4 (up to 4 share a workgroup, more fill
// several).
constexpr int32_t gqa_chunk_waves(int32_t nch) { return nch == 1 ? 1 : (nch == 2 ? 2 : (nch + 3) / 4 * 4); }
// Full blocks per split of the D1 item of `anchor` read by the layers of [l0, l1)
// in table s (split_blocks_for with the item's chunk waves in one workgroup).
int32_t gqa_item_split_blocks(const kvk_table* s, int32_t anchor, int32_t l0, int32_t l1, int32_t n_blocks,
                              int64_t target_bytes, int32_t* count_bound = nullptr);
// Bytes per D1 split for a decode over layers [l0, l1) of a GQA table (see table.cpp).
int64_t gqa_split_target(const kvk_table* t, int32_t l0, int32_t l1);

// Bytes at the head of the workspace that hold the device-side work list of a
// decode over [l0, l1) of a per-sequence table (decode.hip).
int64_t gqa_batched_list_bytes(const kvk_table* t, int32_t l0, int32_t l1);

// Number of decode splits of one stream holding `n_blocks` blocks.
inline int32_t n_splits(int32_t n_blocks, int32_t split_blocks) {
  return (n_blocks + split_blocks - 1) / split_blocks;
}

// ---------------------------------------------------------------------------
// MLA (rank axis)
// ---------------------------------------------------------------------------

// Bytes of one 32-token block of an MLA stream storing W = d + d_R channels.
int64_t mla_block_bytes(int32_t W, int32_t bits, int32_t qscheme);

// MLA decode workgroup geometry for W = d + d_R stored channels: the channel
// parts a 16-token tile is split into (2 for the widest rows), and the 32-token
// blocks one iteration of the four waves covers (16 tokens per tile part).
constexpr int mla_ksplit(int W) { return W > 320 ? 2 : 1; }
constexpr int mla_iter_blocks(int W) { return 2 / mla_ksplit(W); }

// Iterations the MLA decode kernel keeps in flight per workgroup (registers) for
// a stream of W stored channels at `bits`: about 32 KiB of cache, at most 64
// registers per thread (40 from d = 256 on, whose query and accumulators take
// the most).  Shared by the host (split sizes) and the kernel.
constexpr int mla_ring_depth(int W, int bits, int kivi) {
  const int nkw = W / 32 / mla_ksplit(W);                        // k-steps per wave
  const int regs = bits == 16 ? 4 * nkw : (bits == 8 ? 2 * nkw : nkw) + (bits == 16 ? 0 : (kivi ? nkw : 1));
  const long wg_bytes = 4L * 16 * (W / mla_ksplit(W)) * bits / 8;  // codes of one iteration
  const int cap = W > 576 ? 80 : (W > 192 ? 40 : 64);  // width 1024: one wave per SIMD, more registers
  const int by_regs = regs > cap ? 1 : cap / regs;
  const int by_bytes = (int)((32768 + wg_bytes - 1) / wg_bytes);
  const int nr = by_regs < by_bytes ? by_regs : by_bytes;
  return nr < 1 ? 1 : nr;
}

// Query heads of an MLA decode rounded up to whole 16-head tiles (an MFMA's N): the
// absorbed queries and split partials are laid out for this many; the padding heads
// carry zero queries and are never written out.  A decode workgroup takes a chunk
// of two tiles, the last chunk one tile when the padded count is an odd number of
// tiles (40 heads: 32 + 16, not 64).
constexpr int32_t mla_heads_padded(int32_t hq) { return (hq + 15) / 16 * 16; }
constexpr int32_t mla_head_chunks(int32_t hq) { return (mla_heads_padded(hq) + 31) / 32; }

// Most splits of one MLA stream (the merge holds one weight per split in LDS).
constexpr int kMlaMaxUnits = 128;

// Full blocks per split of the MLA decode kernel for an anchor whose streams hold
// n_blocks full blocks: sized so that splits of every width take about the same
// time, balanced over the stream, rounded up to a multiple of the ring depth (so
// only a stream's last split prefetches past its end); the split count is
// monotone in n_blocks.
int32_t mla_split_blocks_for(const kvk_table* t, int32_t anchor, int32_t n_blocks);
// The anchor's split rule in two numbers (mla_split_rule: the target length in
// blocks and the ring pass nr), from which mla_split_len gives the split length for
// any n_blocks; the host and the kernels (which know n_blocks only at decode time
// under per-sequence plans) share it.
void mla_split_rule(const kvk_table* t, int32_t anchor, int32_t* target, int32_t* nr);
constexpr int32_t mla_split_len(int32_t target, int32_t nr, int32_t n_blocks) {
  const int32_t nb = n_blocks > 0 ? n_blocks : 1;
  if ((int64_t)target * kMlaMaxUnits < nb) target = (nb + kMlaMaxUnits - 1) / kMlaMaxUnits;  // merge limit
  const int32_t nsplit = (nb + target - 1) / target;
  const int32_t per = (nb + nsplit - 1) / nsplit;
  return (per + nr - 1) / nr * nr;
}
// At least the splits of every length up to n_blocks_cap full blocks (the partial
// records a workspace sized at the capacity holds).  The split count itself is not
// monotone in the length (rounding a split up to whole ring passes can save one: at
// target 128 blocks and ring pass 6, 2898 blocks take 23 splits and 2899 take 22), but
// it never exceeds the count before that rounding, ceil(n / target), which is.
constexpr int32_t mla_units_bound(int32_t target, int32_t n_blocks_cap) {
  const int32_t nb = n_blocks_cap > 0 ? n_blocks_cap : 1;
  return (int64_t)target * kMlaMaxUnits < nb ? kMlaMaxUnits : (nb + target - 1) / target;
}
// Splits of a stream holding n_stored tokens (n_blocks full ones) with split length
// `split`: the full blocks in balanced splits, the tail in the last; at least one
// unit when anything is stored, none otherwise.
constexpr int32_t mla_units_len(int32_t n_blocks, int32_t n_stored, int32_t split) {
  return n_stored <= 0 ? 0 : (n_blocks > 0 ? (n_blocks + split - 1) / split : 1);
}

// Work units (splits) of one MLA stream holding n_stored tokens: the full blocks
// in balanced splits, the tail tokens in the last one; at least one unit.
int32_t mla_units(const kvk_table* t, int32_t anchor, int32_t n_stored);

// Workspace layout of an MLA decode over [l0, l1): the absorbed queries of each
// layer (fp16 [B][Hq][W]) then the split partials of each layer (fp32, per
// (b, split): m[Hq], l[Hq], o[Hq][d]), each layer's part 256-byte aligned.
// Offsets are sized for the table's capacity.
struct MlaWorkspace {
  int64_t q_off[KVK_MAX_LAYERS];
  int64_t part_off[KVK_MAX_LAYERS];
  int32_t units_cap[KVK_MAX_LAYERS];  // splits per (layer, b) at capacity
  int64_t total;
};
void mla_workspace(const kvk_table* t, int32_t l0, int32_t l1, MlaWorkspace* ws);

kvk_status mla_compress_layer_project(const kvk_table* t, int32_t layer, const void* x, const void* w_dkv,
                                      int32_t d_model, const void* rope, int32_t n_tokens,
                                      const int32_t* keep_idx, void* arena, void* latent_out, hipStream_t stream);
kvk_status mla_compress_layer(const kvk_table* t, int32_t layer, const void* latent,
                              const void* rope, int32_t in_dtype, int32_t n_tokens,
                              const int32_t* keep_idx, void* arena, hipStream_t stream);
// The projected write of one layer of a per-sequence MLA table: one launch per
// (kept width, bit-width) over the sequences whose plans store the layer so.
kvk_status mla_compress_layer_project_batched(const kvk_table* t, int32_t layer, const void* x, const void* w_dkv,
                                              int32_t d_model, const void* rope, int32_t n_tokens,
                                              const int32_t* keep_idx, void* arena, hipStream_t stream);
// The write of one layer of a per-sequence MLA table: one launch per (kept width,
// bit-width) over the sequences whose plans store the layer so.
kvk_status mla_compress_layer_batched(const kvk_table* t, int32_t layer, const void* latent, const void* rope,
                                      int32_t in_dtype, int32_t n_tokens, const int32_t* keep_idx, void* arena,
                                      hipStream_t stream);
kvk_status mla_append_token(const kvk_table* t, int32_t l0, int32_t l1, const void* latent,
                            const void* rope, int32_t in_dtype, int32_t n_stored, void* arena,
                            hipStream_t stream);
// q_lstride / out_lstride: elements between consecutive layers of q / out (0: the
// table's own [B][Hq][...] per layer; a sequence of a per-sequence batch passes the
// batch's, with q and out at its first row).
kvk_status mla_decode_splits(const kvk_table* t, int32_t l0, int32_t l1, const void* q,
                             int32_t q_dtype, int32_t n_stored, float scale, const void* w_uk,
                             const void* arena, void* workspace, hipStream_t stream, int64_t q_lstride = 0);
kvk_status mla_decode_merge(const kvk_table* t, int32_t l0, int32_t l1, int32_t n_stored,
                            const void* w_uv, const void* workspace, float* out,
                            hipStream_t stream, int64_t out_lstride = 0);
// The absorbed queries of `rows` query rows [rows][Hq][nope + d_R] (bf16) at the full
// latent width: out fp16 [rows][Hp][r + d_R], prescaled by scale log2 e (the decode's
// absorption with the window positions of the query-aware keep list as rows).
kvk_status mla_absorb_rows(const kvk_table* t, const void* q, int32_t rows, const void* w_uk, void* out,
                           float scale, hipStream_t stream);
// Per-sequence MLA tables: the work list at the head of the workspace (image when
// `image`; sizes and offsets always).
struct MlaSeqList {
  MlaSeqList();
  ~MlaSeqList();
  std::vector<uint8_t> img;
  int64_t rows_off = 0, items_off[4] = {0, 0, 0, 0}, bytes = 0;
  int32_t n_items[4] = {0, 0, 0, 0};
  int64_t n_wg[4] = {0, 0, 0, 0};
  int32_t dmax = 0;
  uint64_t hash = 0;
};
kvk_status mla_seq_list(const kvk_table* t, int32_t l0, int32_t l1, MlaSeqList& L, bool image);
// One decode of a per-sequence MLA table (A1 + D2 with `splits`, C2 with `merge`):
// one launch per phase for the batch, from the list kvk_decode_setup wrote.
kvk_status mla_decode_batched(const kvk_table* t, int32_t l0, int32_t l1, const void* q, int32_t q_dtype,
                              int32_t n_stored, float scale, const void* w_uk, const void* w_uv,
                              const void* arena, float* out, void* workspace, hipStream_t stream, bool splits,
                              bool merge);
// FNV-1a over n bytes (the work lists' hashes).
uint64_t fnv1a64(const uint8_t* p, size_t n);
kvk_status mla_debug_dequantize(const kvk_table* t, int32_t layer, int32_t n_stored,
                                const void* arena, float* c_out, float* r_out, hipStream_t stream);

}  // namespace kvk
