// plan.h -- host planner of the MSA library (no HIP calls).
#pragma once

#include <string>
#include <vector>

#include "append.h"
#include "msa.h"
#include "msa_internal.h"

namespace msa {

struct HostPlan {
  msa_shape shape{};
  int32_t group = 1;        // G = Hq / Hkv
  int32_t tile_rows = 0;    // rows per tile: kTileRowsDecode, kTileRowsNarrow or kTileRowsWide
  int32_t tile_tokens = 0;  // query tokens per tile
  bool precise_weights = false;  // MSA_PLAN_PRECISE_WEIGHTS: hi + lo weights on every step
  int64_t total_q = 0;
  std::vector<int32_t> row_pos;   // [total_q] absolute position of each packed row
  std::vector<int32_t> seq_blocks; // [num_seqs] block-table entries the plan reads per sequence
  std::vector<WorkItem> work;     // items grouped by workgroup (workgroup i: wg_ptr[i] .. wg_ptr[i+1]-1)
  std::vector<int32_t> wg_ptr;    // [num_workgroups + 1]; workgroup i runs on XCD i % 8
  std::vector<MergeItem> merge;
  std::vector<AppendItem> append; // one per (segment, cache block) slice
  int64_t num_tiles = 0;          // tiles x kv heads before splitting
  int64_t max_splits = 1;
  int64_t num_slots = 0;          // workspace partial slots
  int64_t workspace_bytes = 0;
  double useful_flops = 0, tile_flops = 0, planned_bytes = 0, min_bytes = 0;
};

// Validates the inputs and fills *out.  On error returns the status and a
// message in *err; *out is then unspecified.
msa_status build_plan(const msa_shape* shape, const int32_t* seq_kv_len, const int32_t* seg_indptr,
                      const int32_t* seg_start, const int32_t* seg_len, const msa_plan_opts* opts,
                      HostPlan* out, std::string* err);

}  // namespace msa
