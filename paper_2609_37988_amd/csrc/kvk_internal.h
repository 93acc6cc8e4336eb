// Internal declarations shared by the host-side translation units of libkvk.
#pragma once

#include <cstdarg>
#include <cstdint>
#include <string>

#include "kvk.h"

struct kvk_table {
  kvk_dims d;
  kvk_action plan[KVK_MAX_LAYERS];
  kvk_table_info info;
  int32_t bits[KVK_MAX_LAYERS];         // bits of each layer's own action (anchors)
  int64_t block_bytes[KVK_MAX_LAYERS];  // bytes of one 32-token block (anchors)
  int32_t next_anchor[KVK_MAX_LAYERS];  // first anchor after l (n_layers if none)
  int32_t cap;                          // stored tokens capacity per stream
  int32_t nb_cap;                       // full-block capacity per stream (cap / 32)
};

namespace kvk {

// Thread-local last-error message.
void set_error(const char* fmt, ...);
kvk_status fail(kvk_status st, const char* fmt, ...);

inline int64_t round256(int64_t n) { return (n + 255) / 256 * 256; }

// Bytes of one 32-token block of a GQA stream with `bits`-bit codes.
int64_t gqa_block_bytes(int32_t head_dim, int32_t bits, int32_t qscheme);

// Blocks the decode kernel keeps in flight per wave for a `bits`-bit anchor
// (must equal the kernel's ring depth).
int32_t ring_depth_for(int32_t bits);

// Blocks processed per split of the decode kernel for a `bits`-bit anchor whose
// streams hold n_blocks full blocks.  The split count never exceeds the one at a
// larger n_blocks, so workspace sized at capacity covers every n_stored.
int32_t split_blocks_for(int32_t bits, int32_t qscheme, int32_t head_dim, int32_t n_blocks);

// Number of decode splits of one stream holding `n_blocks` blocks.
inline int32_t n_splits(int32_t n_blocks, int32_t split_blocks) {
  return (n_blocks + split_blocks - 1) / split_blocks;
}

}  // namespace kvk
