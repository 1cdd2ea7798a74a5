// append.h -- arguments and launcher of the paged K/V append kernel.
//
// The query tokens of all segments run through one forward pass (Sec. 4.1),
// so each layer produces the fresh keys and values of every packed row; they
// go into the paged cache (Sec. 5.3: the cache is PagedAttention's) at the
// row's absolute position before the attention reads them.
#pragma once

#include <cstdint>

namespace msa {

// One workgroup of the append: the rows of one segment that fall into one
// cache block (consecutive rows row0 .. row0+n-1 at positions pos0 .. pos0+n-1,
// 1 <= n <= 16, all inside block pos0 / 16 of sequence seq).
struct AppendItem {
  int32_t row0;
  int32_t seq;
  int32_t pos0;
  int32_t n;
};
static_assert(sizeof(AppendItem) == 16, "AppendItem is 4 int32");

struct AppendParams {
  const uint16_t* k_new;      // [total_q, Hkv, d] strided
  const uint16_t* v_new;
  const int32_t* block_table; // [num_seqs * max_blocks]
  const AppendItem* items;
  uint16_t* k_cache;
  uint16_t* v_cache;
  int64_t kn_st, kn_sh, vn_st, vn_sh;
  int64_t k_sb, k_sh, k_st;
  int64_t v_sb, v_sh, v_sd;
  int32_t num_kv_heads;
  int32_t max_blocks;
  int32_t num_blocks;
};

// Returns a hipError_t value as int.
int launch_kv_append(const AppendParams& p, int head_dim, int num_items, void* stream);

}  // namespace msa
