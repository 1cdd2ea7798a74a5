// api.cpp -- the C ABI declared in include/msa.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "msa.h"
#include "append.h"
#include "errors.h"
#include "forward.h"
#include "msa_internal.h"
#include "plan.h"

struct msa_plan_s {
  msa::HostPlan hp;
  bool host_only = true;
  int device = -1;
  std::vector<char> staging;  // host image of the device buffer (kept alive for the async copy)
  char* dev = nullptr;        // device buffer: row_pos | work | merge | append | wg_ptr
  const int32_t* d_row_pos = nullptr;
  const msa::WorkItem* d_work = nullptr;
  const int32_t* d_wg_ptr = nullptr;
  const msa::MergeItem* d_merge = nullptr;
  const msa::AppendItem* d_append = nullptr;
};

namespace {

thread_local std::string g_last_error;

msa_status set_error(msa_status st, const std::string& msg) {
  g_last_error = msg;
  return st;
}

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

}  // namespace

void msa::set_last_error(const std::string& msg) { g_last_error = msg; }

msa_status msa::forward_impl(const char* who, msa_plan_t plan, const void* q, const void* k_cache,
                        const void* v_cache, const int32_t* block_table, void* o, float* lse,
                        void* workspace, size_t workspace_bytes, void* hip_stream) {
  const std::string w(who);
  if (!plan) return set_error(MSA_ERR_INVALID_ARG, w + ": null plan");
  if (plan->host_only)
    return set_error(MSA_ERR_INVALID_ARG, w + ": plan was built with MSA_PLAN_HOST_ONLY");
  const msa::HostPlan& hp = plan->hp;
  if (hp.work.empty()) return MSA_OK;  // no query rows: nothing to do
  if (!q || !k_cache || !v_cache || !block_table || !o)
    return set_error(MSA_ERR_INVALID_ARG, w + ": q, k_cache, v_cache, block_table, o must be non-null");
  if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(o, 16) ||
      !aligned(block_table, 4) || (lse && !aligned(lse, 4)))
    return set_error(MSA_ERR_INVALID_ARG, w + ": q/k/v/o must be 16-byte aligned");
  if ((size_t)hp.workspace_bytes > workspace_bytes)
    return set_error(MSA_ERR_INVALID_ARG,
                     w + ": workspace too small (need " + std::to_string(hp.workspace_bytes) +
                         " bytes)");
  if (hp.workspace_bytes > 0 && (!workspace || !aligned(workspace, 16)))
    return set_error(MSA_ERR_INVALID_ARG, w + ": workspace must be non-null and 16-byte aligned");
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != plan->device)
    return set_error(MSA_ERR_INVALID_ARG, w + ": current device differs from the plan's device");

  const msa_shape& s = hp.shape;
  msa::AttnParams p{};
  p.q = static_cast<const uint16_t*>(q);
  p.k = static_cast<const uint16_t*>(k_cache);
  p.v = static_cast<const uint16_t*>(v_cache);
  p.block_table = block_table;
  p.row_pos = plan->d_row_pos;
  p.work = plan->d_work;
  p.wg_ptr = plan->d_wg_ptr;
  p.o = static_cast<uint16_t*>(o);
  p.lse = lse;
  p.ws = static_cast<float*>(workspace);
  p.q_st = s.q_stride_tok;
  p.q_sh = s.q_stride_head;
  p.o_st = s.o_stride_tok;
  p.o_sh = s.o_stride_head;
  p.k_sb = s.k_stride_block;
  p.k_sh = s.k_stride_head;
  p.k_st = s.k_stride_tok;
  p.v_sb = s.v_stride_block;
  p.v_sh = s.v_stride_head;
  p.v_sd = s.v_stride_dim;
  p.max_blocks = s.max_blocks_per_seq;
  p.num_q_heads = s.num_q_heads;
  p.group = hp.group;
  p.tile_tokens = hp.tile_tokens;
  p.scale_log2 = s.scale * 1.4426950408889634f;
  p.precise = hp.precise_weights ? 1 : 0;
  const int num_wg = hp.wg_ptr.empty() ? 0 : (int)hp.wg_ptr.size() - 1;
  int rc = msa::launch_attn(p, s.head_dim, hp.tile_rows, num_wg, hip_stream);
  if (rc != 0) return set_error(MSA_ERR_DEVICE, std::string(w + ": attention launch failed: ") +
                                                    hipGetErrorString((hipError_t)rc));
  if (!hp.merge.empty()) {
    msa::MergeParams m{};
    m.merge = plan->d_merge;
    m.ws = static_cast<const float*>(workspace);
    m.o = static_cast<uint16_t*>(o);
    m.lse = lse;
    m.o_st = s.o_stride_tok;
    m.o_sh = s.o_stride_head;
    m.num_q_heads = s.num_q_heads;
    m.group = hp.group;
    m.tile_rows = hp.tile_rows;
    rc = msa::launch_merge(m, s.head_dim, (int)hp.merge.size(), hip_stream);
    if (rc != 0) return set_error(MSA_ERR_DEVICE, std::string(w + ": merge launch failed: ") +
                                                      hipGetErrorString((hipError_t)rc));
  }
  return MSA_OK;
}

int64_t msa::plan_workspace_bytes(msa_plan_t plan) { return plan->hp.workspace_bytes; }

extern "C" {

const char* msa_last_error(void) { return g_last_error.c_str(); }

msa_status msa_plan(const msa_shape* shape, const int32_t* seq_kv_len, const int32_t* seg_indptr,
                    const int32_t* seg_start, const int32_t* seg_len, const msa_plan_opts* opts,
                    void* hip_stream, msa_plan_t* out) {
  if (!out) return set_error(MSA_ERR_INVALID_ARG, "msa_plan: out must be non-null");
  *out = nullptr;
  msa_plan_s* plan = new (std::nothrow) msa_plan_s();
  if (!plan) return set_error(MSA_ERR_OUT_OF_MEMORY, "msa_plan: host allocation failed");
  std::string err;
  msa_status st;
  try {
    st = msa::build_plan(shape, seq_kv_len, seg_indptr, seg_start, seg_len, opts, &plan->hp, &err);
  } catch (const std::bad_alloc&) {
    st = MSA_ERR_OUT_OF_MEMORY;
    err = "host allocation failed while planning";
  }
  if (st != MSA_OK) {
    delete plan;
    return set_error(st, "msa_plan: " + err);
  }
  plan->host_only = opts && (opts->flags & MSA_PLAN_HOST_ONLY);
  if (!plan->host_only) {
    const msa::HostPlan& hp = plan->hp;
    const size_t n_row = hp.row_pos.size() * sizeof(int32_t);
    const size_t n_work = hp.work.size() * sizeof(msa::WorkItem);
    const size_t n_merge = hp.merge.size() * sizeof(msa::MergeItem);
    const size_t n_append = hp.append.size() * sizeof(msa::AppendItem);
    const size_t n_wg = hp.wg_ptr.size() * sizeof(int32_t);
    const size_t off_work = align_up(n_row, 256);
    const size_t off_merge = off_work + align_up(n_work, 256);
    const size_t off_append = off_merge + align_up(n_merge, 256);
    const size_t off_wg = off_append + align_up(n_append, 256);
    const size_t bytes = std::max<size_t>(off_wg + n_wg, 256);
    try {
      plan->staging.assign(bytes, 0);
    } catch (const std::bad_alloc&) {
      delete plan;
      return set_error(MSA_ERR_OUT_OF_MEMORY, "msa_plan: host allocation failed");
    }
    if (n_row) std::memcpy(plan->staging.data(), hp.row_pos.data(), n_row);
    if (n_work) std::memcpy(plan->staging.data() + off_work, hp.work.data(), n_work);
    if (n_merge) std::memcpy(plan->staging.data() + off_merge, hp.merge.data(), n_merge);
    if (n_append) std::memcpy(plan->staging.data() + off_append, hp.append.data(), n_append);
    if (n_wg) std::memcpy(plan->staging.data() + off_wg, hp.wg_ptr.data(), n_wg);
    const hipError_t gd = hipGetDevice(&plan->device);
    if (gd != hipSuccess) {
      delete plan;
      return set_error(MSA_ERR_DEVICE, std::string("msa_plan: hipGetDevice failed: ") + hipGetErrorString(gd));
    }
    void* dev = nullptr;
    if (hipMalloc(&dev, bytes) != hipSuccess) {
      (void)hipGetLastError();
      delete plan;
      return set_error(MSA_ERR_OUT_OF_MEMORY, "msa_plan: hipMalloc of the plan buffer failed");
    }
    plan->dev = static_cast<char*>(dev);
    if (hipMemcpyAsync(dev, plan->staging.data(), bytes, hipMemcpyHostToDevice,
                       static_cast<hipStream_t>(hip_stream)) != hipSuccess) {
      (void)hipGetLastError();
      (void)hipFree(dev);
      delete plan;
      return set_error(MSA_ERR_DEVICE, "msa_plan: upload of the plan buffer failed");
    }
    plan->d_row_pos = reinterpret_cast<const int32_t*>(plan->dev);
    plan->d_work = reinterpret_cast<const msa::WorkItem*>(plan->dev + off_work);
    plan->d_merge = reinterpret_cast<const msa::MergeItem*>(plan->dev + off_merge);
    plan->d_wg_ptr = reinterpret_cast<const int32_t*>(plan->dev + off_wg);
    plan->d_append = reinterpret_cast<const msa::AppendItem*>(plan->dev + off_append);
  }
  *out = plan;
  return MSA_OK;
}

msa_status msa_plan_info(msa_plan_t plan, msa_plan_info_t* info) {
  if (!plan || !info) return set_error(MSA_ERR_INVALID_ARG, "msa_plan_info: null argument");
  const msa::HostPlan& hp = plan->hp;
  info->total_q = hp.total_q;
  info->num_work = (int64_t)hp.work.size();
  info->num_tiles = hp.num_tiles;
  info->num_merge = (int64_t)hp.merge.size();
  info->max_splits = hp.max_splits;
  info->workspace_bytes = hp.workspace_bytes;
  info->useful_flops = hp.useful_flops;
  info->tile_flops = hp.tile_flops;
  info->planned_bytes = hp.planned_bytes;
  info->min_bytes = hp.min_bytes;
  info->tile_rows = hp.tile_rows;
  info->num_workgroups = hp.wg_ptr.empty() ? 0 : (int64_t)hp.wg_ptr.size() - 1;
  return MSA_OK;
}

msa_status msa_plan_export(msa_plan_t plan, int32_t* row_pos, int32_t* work, int32_t* merge) {
  if (!plan) return set_error(MSA_ERR_INVALID_ARG, "msa_plan_export: null plan");
  const msa::HostPlan& hp = plan->hp;
  if (row_pos && !hp.row_pos.empty())
    std::memcpy(row_pos, hp.row_pos.data(), hp.row_pos.size() * sizeof(int32_t));
  if (work && !hp.work.empty())
    std::memcpy(work, hp.work.data(), hp.work.size() * sizeof(msa::WorkItem));
  if (merge && !hp.merge.empty())
    std::memcpy(merge, hp.merge.data(), hp.merge.size() * sizeof(msa::MergeItem));
  return MSA_OK;
}

void msa_plan_destroy(msa_plan_t plan) {
  if (!plan) return;
  if (plan->dev) (void)hipFree(plan->dev);
  delete plan;
}

msa_status msa_forward(msa_plan_t plan, const void* q, const void* k_cache, const void* v_cache,
                       const int32_t* block_table, void* o, float* lse, void* workspace,
                       size_t workspace_bytes, void* hip_stream) {
  return msa::forward_impl("msa_forward", plan, q, k_cache, v_cache, block_table, o, lse, workspace,
                           workspace_bytes, hip_stream);
}

msa_status msa_check_block_table(msa_plan_t plan, const int32_t* block_table, int32_t location,
                                 void* hip_stream) {
  if (!plan) return set_error(MSA_ERR_INVALID_ARG, "msa_check_block_table: null plan");
  if (location != MSA_TABLE_HOST && location != MSA_TABLE_DEVICE)
    return set_error(MSA_ERR_INVALID_ARG, "msa_check_block_table: location must be MSA_TABLE_HOST or MSA_TABLE_DEVICE");
  const msa::HostPlan& hp = plan->hp;
  const msa_shape& s = hp.shape;
  int32_t width = 0;  // entries read per row: the most any sequence needs
  for (int32_t nb : hp.seq_blocks) width = std::max(width, nb);
  if (width == 0) return MSA_OK;  // the plan reads no entry
  if (!block_table) return set_error(MSA_ERR_INVALID_ARG, "msa_check_block_table: null block_table");
  if (!aligned(block_table, 4))
    return set_error(MSA_ERR_INVALID_ARG, "msa_check_block_table: block_table must be 4-byte aligned");
  const int32_t* table = block_table;
  std::vector<int32_t> host;
  if (location == MSA_TABLE_DEVICE) {
    try {
      host.assign((size_t)s.num_seqs * (size_t)width, 0);
    } catch (const std::bad_alloc&) {
      return set_error(MSA_ERR_OUT_OF_MEMORY, "msa_check_block_table: host allocation failed");
    }
    // the first `width` entries of every row, in one strided copy
    hipStream_t st = static_cast<hipStream_t>(hip_stream);
    hipError_t e = hipMemcpy2DAsync(host.data(), (size_t)width * sizeof(int32_t), block_table,
                                    (size_t)s.max_blocks_per_seq * sizeof(int32_t),
                                    (size_t)width * sizeof(int32_t), (size_t)s.num_seqs,
                                    hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return set_error(MSA_ERR_DEVICE, std::string("msa_check_block_table: copy of the table failed: ") +
                                           hipGetErrorString(e));
    }
    table = host.data();
  }
  const int64_t row_stride = location == MSA_TABLE_DEVICE ? width : s.max_blocks_per_seq;
  for (int32_t b = 0; b < s.num_seqs; ++b) {
    const int32_t* row = table + (int64_t)b * row_stride;
    for (int32_t i = 0; i < hp.seq_blocks[(size_t)b]; ++i)
      if (row[i] < 0 || row[i] >= s.num_blocks)
        return set_error(MSA_ERR_INVALID_ARG,
                         "msa_check_block_table: sequence " + std::to_string(b) + ", logical block " +
                             std::to_string(i) + " maps to physical block " + std::to_string(row[i]) +
                             ", outside [0, " + std::to_string(s.num_blocks) + ")");
  }
  return MSA_OK;
}

msa_status msa_kv_append(msa_plan_t plan, const void* k_new, const void* v_new,
                         int64_t k_new_stride_tok, int64_t k_new_stride_head,
                         int64_t v_new_stride_tok, int64_t v_new_stride_head,
                         const int32_t* block_table, void* k_cache, void* v_cache,
                         void* hip_stream) {
  if (!plan) return set_error(MSA_ERR_INVALID_ARG, "msa_kv_append: null plan");
  auto ok_stride = [](int64_t x) { return x > 0 && x % 8 == 0; };
  if (!ok_stride(k_new_stride_tok) || !ok_stride(k_new_stride_head) ||
      !ok_stride(v_new_stride_tok) || !ok_stride(v_new_stride_head))
    return set_error(MSA_ERR_INVALID_ARG,
                     "msa_kv_append: strides must be positive multiples of 8 elements");
  if (plan->host_only)
    return set_error(MSA_ERR_INVALID_ARG, "msa_kv_append: plan was built with MSA_PLAN_HOST_ONLY");
  const msa::HostPlan& hp = plan->hp;
  const msa_shape& s = hp.shape;
  if (hp.total_q == 0) return MSA_OK;  // no query rows: nothing to write
  if (!k_new || !v_new || !block_table || !k_cache || !v_cache)
    return set_error(MSA_ERR_INVALID_ARG,
                     "msa_kv_append: k_new, v_new, block_table, k_cache, v_cache must be non-null");
  if (!aligned(k_new, 16) || !aligned(v_new, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) ||
      !aligned(block_table, 4))
    return set_error(MSA_ERR_INVALID_ARG, "msa_kv_append: k/v pointers must be 16-byte aligned");
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != plan->device)
    return set_error(MSA_ERR_INVALID_ARG, "msa_kv_append: current device differs from the plan's device");
  msa::AppendParams p{};
  p.k_new = static_cast<const uint16_t*>(k_new);
  p.v_new = static_cast<const uint16_t*>(v_new);
  p.block_table = block_table;
  p.items = plan->d_append;
  p.k_cache = static_cast<uint16_t*>(k_cache);
  p.v_cache = static_cast<uint16_t*>(v_cache);
  p.kn_st = k_new_stride_tok;
  p.kn_sh = k_new_stride_head;
  p.vn_st = v_new_stride_tok;
  p.vn_sh = v_new_stride_head;
  p.k_sb = s.k_stride_block;
  p.k_sh = s.k_stride_head;
  p.k_st = s.k_stride_tok;
  p.v_sb = s.v_stride_block;
  p.v_sh = s.v_stride_head;
  p.v_sd = s.v_stride_dim;
  p.num_kv_heads = s.num_kv_heads;
  p.max_blocks = s.max_blocks_per_seq;
  p.num_blocks = s.num_blocks;
  const int rc = msa::launch_kv_append(p, s.head_dim, (int)hp.append.size(), hip_stream);
  if (rc != 0)
    return set_error(MSA_ERR_DEVICE, std::string("msa_kv_append: launch failed: ") +
                                         hipGetErrorString((hipError_t)rc));
  return MSA_OK;
}

}  // extern "C"
