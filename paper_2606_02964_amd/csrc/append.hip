// append.hip -- gfx950 kernel that writes the fresh K/V of the packed query
// rows into their paged cache slots.
//
// One workgroup (256 threads) takes one slice: the n <= 16 consecutive rows
// of one segment that land in one cache block (the planner cuts every segment
// at block boundaries), for every KV head, eight heads per pass:
//   * K blocks are token-major, so each (row, head) is one contiguous d-vector
//     in both the source and the cache: 16-byte loads and stores, 16 lanes per
//     row (256 contiguous bytes for d = 128).
//   * V blocks are channel-major (the 16 tokens of one channel are adjacent),
//     so the slice is staged in LDS and written out per channel.  A half block
//     (tokens 0-7 or 8-15) that the slice covers entirely is written as one
//     16-byte store per channel; a partly covered half (the first and last
//     block of a segment) is written token by token with consecutive lanes on
//     consecutive tokens of one channel.
// A slice whose block-table entry is outside [0, num_blocks) is not written.
// The kernel is bound by HBM: it reads and writes each fresh K/V byte once.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "append.h"

namespace msa {
namespace {

constexpr int kHeadsPerPass = 8;

template <int D>
__global__ __launch_bounds__(256) void msa_kv_append_kernel(AppendParams p) {
  constexpr int kChunks = D / 8;  // 16-byte chunks of one head vector
  constexpr int kPitch = D + 8;   // LDS row pitch (elements), breaks bank aliasing
  __shared__ __align__(16) uint16_t s_v[kHeadsPerPass][16][kPitch];

  const uint16_t* __restrict__ k_new = p.k_new;
  const uint16_t* __restrict__ v_new = p.v_new;
  uint16_t* __restrict__ k_cache = p.k_cache;
  uint16_t* __restrict__ v_cache = p.v_cache;

  const AppendItem it = p.items[blockIdx.x];
  const int32_t blk = p.block_table[(int64_t)it.seq * p.max_blocks + it.pos0 / 16];
  if (blk < 0 || blk >= p.num_blocks) return;  // uniform over the workgroup
  const int off0 = it.pos0 % 16;                // slice = tokens off0 .. off0+n-1 of the block
  const int n = it.n;
  const int tid = threadIdx.x;
  const int64_t kbase = (int64_t)blk * p.k_sb;
  const int64_t vbase = (int64_t)blk * p.v_sb;

  for (int g0 = 0; g0 < p.num_kv_heads; g0 += kHeadsPerPass) {
    const int ng = p.num_kv_heads - g0 < kHeadsPerPass ? p.num_kv_heads - g0 : kHeadsPerPass;
    // K straight to the cache; V rows into LDS (slice row i at LDS row off0 + i).
    for (int idx = tid; idx < ng * n * kChunks; idx += 256) {
      const int ch = idx % kChunks;
      const int i = (idx / kChunks) % n;
      const int gl = idx / (kChunks * n);
      const int64_t g = g0 + gl;
      const int64_t r = (int64_t)it.row0 + i;
      const uint4 kv = *reinterpret_cast<const uint4*>(k_new + r * p.kn_st + g * p.kn_sh + ch * 8);
      const uint4 vv = *reinterpret_cast<const uint4*>(v_new + r * p.vn_st + g * p.vn_sh + ch * 8);
      *reinterpret_cast<uint4*>(k_cache + kbase + g * p.k_sh + (int64_t)(off0 + i) * p.k_st +
                                ch * 8) = kv;
      *reinterpret_cast<uint4*>(&s_v[gl][off0 + i][ch * 8]) = vv;
    }
    __syncthreads();
    // V out, one half block (8 tokens) at a time.
    for (int h = 0; h < 2; ++h) {
      const int lo = off0 > 8 * h ? off0 : 8 * h;
      const int hi = off0 + n < 8 * h + 8 ? off0 + n : 8 * h + 8;
      if (lo >= hi) continue;  // the slice misses this half
      if (lo == 8 * h && hi == 8 * h + 8) {
        for (int idx = tid; idx < ng * D; idx += 256) {
          const int c = idx % D;
          const int gl = idx / D;
          uint32_t w[4];
#pragma unroll
          for (int t = 0; t < 4; ++t)
            w[t] = (uint32_t)s_v[gl][8 * h + 2 * t][c] | ((uint32_t)s_v[gl][8 * h + 2 * t + 1][c] << 16);
          *reinterpret_cast<uint4*>(v_cache + vbase + (int64_t)(g0 + gl) * p.v_sh +
                                    (int64_t)c * p.v_sd + 8 * h) = make_uint4(w[0], w[1], w[2], w[3]);
        }
      } else {
        const int w = hi - lo;
        for (int idx = tid; idx < ng * D * w; idx += 256) {
          const int t = lo + idx % w;
          const int c = (idx / w) % D;
          const int gl = idx / (w * D);
          v_cache[vbase + (int64_t)(g0 + gl) * p.v_sh + (int64_t)c * p.v_sd + t] = s_v[gl][t][c];
        }
      }
    }
    __syncthreads();
  }
}

}  // namespace

int launch_kv_append(const AppendParams& p, int head_dim, int num_items, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (num_items <= 0) return 0;
  if (head_dim == 128)
    hipLaunchKernelGGL(msa_kv_append_kernel<128>, dim3(num_items), dim3(256), 0, s, p);
  else if (head_dim == 64)
    hipLaunchKernelGGL(msa_kv_append_kernel<64>, dim3(num_items), dim3(256), 0, s, p);
  else
    return (int)hipErrorInvalidValue;
  return (int)hipGetLastError();
}

}  // namespace msa
