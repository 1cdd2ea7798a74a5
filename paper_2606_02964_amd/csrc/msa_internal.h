// msa_internal.h -- tables shared by the host planner and the gfx950 kernels.
//
// A work item is one tile: up to tile_rows query rows of one sequence
// that share one KV head (tokens x the G = Hq/Hkv query heads of the group,
// row r <-> token r / G, head r % G) and one contiguous key range.  The
// launch is persistent: each workgroup runs its own list of items.  The
// planner packs consecutive query tokens of a sequence into a tile even
// across segment gaps; each row keeps its own causal limit (its absolute
// position), which is what the paper's per-token "equivalent seq_len" array
// provides (Sec. 4.1).
#pragma once

#include <cstdint>

namespace msa {

// Tile widths: 128 rows (4 waves x 32 rows, two workgroups per CU) for
// small plans, 256 rows (8 waves, one workgroup per CU) for plans with many
// tiles (a wider tile loads each K/V step once for twice the rows), and 32
// rows for decode-like plans (every tile holds at most 32 rows; the four
// waves split the tile's keys and read K/V straight into registers).
constexpr int kTileRowsNarrow = 128;
constexpr int kTileRowsWide = 256;
constexpr int kTileRowsDecode = 32;
constexpr int kKvStep = 64;      // keys per main-loop iteration (4 blocks of 16)
constexpr int kBlockSize = 16;

struct WorkItem {
  int32_t seq;
  int32_t kv_head;
  int32_t row0;      // first packed token row
  int32_t nrows;     // tokens in the tile; 0 = empty padding item
  int32_t kv_lo;     // first key (multiple of kKvStep)
  int32_t kv_hi;     // one past the last key
  int32_t out_slot;  // -1: final output; >= 0: workspace slot of a partial
  int32_t wg;        // the workgroup (blockIdx.x) that runs it
};
static_assert(sizeof(WorkItem) == 32, "WorkItem is exported as 8 int32");

struct MergeItem {
  int32_t seq;
  int32_t kv_head;
  int32_t row0;
  int32_t nrows;
  int32_t nsplit;
  int32_t slot0;     // partial slots slot0 .. slot0 + nsplit - 1, in key order
  int32_t pad0, pad1;
};
static_assert(sizeof(MergeItem) == 32, "MergeItem is exported as 8 int32");

// Workspace slot of one partial tile result: O [tile_rows][d] fp32 (already
// divided by its own softmax sum), then lse [tile_rows] fp32 (natural log).
inline int64_t slot_floats(int head_dim, int tile_rows) { return (int64_t)tile_rows * (head_dim + 1); }

// Arguments of the attention kernel.
struct AttnParams {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* block_table;
  const int32_t* row_pos;
  const WorkItem* work;
  const int32_t* wg_ptr;  // workgroup i runs items wg_ptr[i] .. wg_ptr[i+1]-1, in order
  uint16_t* o;
  float* lse;        // may be null
  float* ws;         // workspace (partials), may be null when unused
  int64_t q_st, q_sh, o_st, o_sh;
  int64_t k_sb, k_sh, k_st;
  int64_t v_sb, v_sh, v_sd;
  int32_t max_blocks;
  int32_t num_q_heads;
  int32_t group;     // G = Hq / Hkv
  int32_t tile_tokens;
  float scale_log2;  // scale * log2(e)
  int32_t precise;   // nonzero: every step carries hi + lo weights (MSA_PLAN_PRECISE_WEIGHTS)
};

struct MergeParams {
  const MergeItem* merge;
  const float* ws;
  uint16_t* o;
  float* lse;
  int64_t o_st, o_sh;
  int32_t num_q_heads;
  int32_t group;
  int32_t tile_rows;  // rows of a workspace slot
};

// Launchers (attn.hip).  Return a hipError_t value as int.
int launch_attn(const AttnParams& p, int head_dim, int tile_rows, int num_wg, void* stream);
int launch_merge(const MergeParams& p, int head_dim, int num_merge, void* stream);

}  // namespace msa
