// attn.hip -- gfx950 kernels of Multi-Segment Attention.
//
// msa_attn: one workgroup per work item = up to 32 rows per wave (4 or 8
// waves: 128 or 256 rows) of one sequence sharing one KV head, over one key
// range.  The wide form loads each K/V step once for twice the rows (one
// workgroup per CU); the narrow form keeps two workgroups per CU for small
// plans.  Per 64-key step:
//   - paged gather: the 4 cache blocks of the step are looked up in the block
//     table and copied to LDS with 16-byte loads (K as [key][d], V as [d][key]
//     since the V cache is channel-major inside a block), double buffered;
//   - S^T = K Q^T on v_mfma_f32_32x32x16_bf16.  K is the A operand, so in the
//     result each lane holds one query row (column) and 16 of the 32 keys:
//     row max and row sum need one exchange with the lane 32 apart only;
//   - per-row causal limit: key j is visible to the row at absolute position
//     p iff j <= p (applied only on steps that reach past the smallest
//     position of the wave);
//   - online softmax in fp32 in the exp2 domain: the row max is taken on the
//     raw scores, scale * log2(e) enters one FMA per score; the reference max
//     only moves (and O is only rescaled) when a row's max grows by more than
//     2^8, so most steps skip the rescale; the row sum adds the bf16-rounded
//     weights with v_dot2 against (1, 1);
//   - O^T += V^T P^T on the same MFMA: P is the B operand and is packed to
//     bf16 straight from the score registers.  The A-operand row order of K is
//     permuted (bits 2 and 3 of the row index swapped) so that the 8 scores a
//     lane feeds to one PV step are 8 consecutive keys, matching a single
//     16-byte LDS read of V^T.
// msa_merge: combines the per-split partials of a split tile by log-sum-exp.
#include <hip/hip_runtime.h>

#include <climits>
#include <cstdint>
#include <type_traits>

#include "msa_internal.h"

namespace msa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kLn2 = 0.69314718055994531f;
constexpr float kLog2e = 1.4426950408889634f;

template <int D>
struct Tile {
  static constexpr int kPitchK = D * 2 + 16;        // bytes per key row of the K tile
  static constexpr int kPitchV = kKvStep * 2 + 16;  // bytes per channel row of the V^T tile
  static constexpr int kBytesK = kKvStep * kPitchK;
  static constexpr int kBytesV = D * kPitchV;
  static constexpr int kStage = kBytesK + kBytesV;
};

__device__ __forceinline__ int swap_bits23(int m) {
  return (m & ~12) | ((m & 4) << 1) | ((m & 8) >> 1);
}

// max / sum of x over the lane pair (l, l ^ 32)
__device__ __forceinline__ float pair_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// bf16 pair (a, b) packed into one register, round to nearest even
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  const bf16x2 v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

// running-max threshold of the lazy rescale: the reference max only moves
// when a row's max grows by more than this (log2 units), so the unnormalised
// weights stay <= 2^8
constexpr float kRescaleLog2 = 8.0f;

template <int D, int W>
__global__ __launch_bounds__(64 * W, 2) void msa_attn_kernel(AttnParams p) {
  using T = Tile<D>;
  constexpr int kThreads = 64 * W;
  constexpr int kRows = 32 * W;                          // tile rows
  constexpr int kRounds = kKvStep * D / 8 / kThreads;    // 16-byte chunks per thread, per tensor
  __shared__ __attribute__((aligned(16))) char smem[2 * T::kStage];

  const WorkItem w = p.work[blockIdx.x];
  if (w.nrows == 0) return;  // padding item (uniform over the workgroup)

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63, hl = lane >> 5, ln = lane & 31;
  const int G = p.group;
  const int r = wave * 32 + ln;  // tile row
  const int t = r / G, hh = r - t * G;
  const bool valid = t < w.nrows;
  const int tok = w.row0 + t;
  const int head = w.kv_head * G + hh;
  const int pos = valid ? p.row_pos[tok] : -1;

  // wave-wide smallest and largest causal limit (wave-uniform branches)
  int pmin = valid ? pos : INT_MAX, pmax = pos;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    pmin = min(pmin, __shfl_xor(pmin, off));
    pmax = max(pmax, __shfl_xor(pmax, off));
  }

  // Q fragments (B operand): row r, channels kk*16 + hl*8 .. +8
  bf16x8 qf[D / 16];
  {
    const uint16_t* qrow = p.q + (int64_t)tok * p.q_st + (int64_t)head * p.q_sh + hl * 8;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      if (valid) {
        qf[kk] = *reinterpret_cast<const bf16x8*>(qrow + kk * 16);
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) qf[kk][j] = (__bf16)0.0f;
      }
    }
  }

  // Gather geometry.  One cache block of one KV head is 16 keys x D
  // channels = 2*D chunks of 16 bytes per tensor; the workgroup's threads
  // cover kThreads / (2*D) blocks per round, kRounds rounds cover the 4
  // blocks of a step.  Thread tid takes chunk cb = tid % (2*D) of block
  // i * (kThreads / (2*D)) + tid / (2*D) in round i.
  constexpr int kChunksPerBlock = 2 * D;
  constexpr int kBlocksPerRound = kThreads / kChunksPerBlock;
  const int cb = tid % kChunksPerBlock;
  const int bsub = tid / kChunksPerBlock;  // wave-uniform
  const int kkey = cb / (D / 8), kdch = cb % (D / 8);
  const int vch = cb >> 1, vhalf = cb & 1;
  const uint32_t koff = (uint32_t)(kkey * p.k_st + kdch * 8) * 2u;   // bytes inside a block
  const uint32_t voff = (uint32_t)(vch * p.v_sd + vhalf * 8) * 2u;
  const int64_t ksb = p.k_sb * 2, vsb = p.v_sb * 2;                   // bytes per block
  const char* kbase = reinterpret_cast<const char*>(p.k + (int64_t)w.kv_head * p.k_sh);
  const char* vbase = reinterpret_cast<const char*>(p.v + (int64_t)w.kv_head * p.v_sh);
  const int32_t* bt = p.block_table + (int64_t)w.seq * p.max_blocks;
  int klds[kRounds], vlds[kRounds];
#pragma unroll
  for (int i = 0; i < kRounds; ++i) {
    const int blk = i * kBlocksPerRound + bsub;
    klds[i] = (blk * 16 + kkey) * T::kPitchK + kdch * 16;
    vlds[i] = T::kBytesK + vch * T::kPitchV + (blk * 16 + vhalf * 8) * 2;
  }

  uint4 kr[kRounds], vr[kRounds];
  // global -> registers for the step starting at key kb; blocks at or past
  // kv_hi are not read (their block-table entries need not be valid)
  auto load = [&](int kb) {
    int ids[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) ids[j] = kb + j * kBlockSize < w.kv_hi ? bt[(kb >> 4) + j] : -1;
#pragma unroll
    for (int i = 0; i < kRounds; ++i) {
      const int id = kBlocksPerRound == 1 ? ids[i] : ids[i * kBlocksPerRound + bsub];
      if (id >= 0) {
        kr[i] = *reinterpret_cast<const uint4*>(kbase + id * ksb + koff);
        vr[i] = *reinterpret_cast<const uint4*>(vbase + id * vsb + voff);
      } else {
        kr[i] = make_uint4(0, 0, 0, 0);
        vr[i] = make_uint4(0, 0, 0, 0);
      }
    }
  };
  auto store = [&](char* st) {
#pragma unroll
    for (int i = 0; i < kRounds; ++i) {
      *reinterpret_cast<uint4*>(st + klds[i]) = kr[i];
      *reinterpret_cast<uint4*>(st + vlds[i]) = vr[i];
    }
  };

  const float c = p.scale_log2;  // > 0
  float m_ref = -__builtin_inff(), l_run = 0.0f;
  f32x16 oacc[D / 32];
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int i = 0; i < 16; ++i) oacc[dt][i] = 0.0f;
  const int klane = swap_bits23(ln) * T::kPitchK + hl * 16;
  const int vlane = T::kBytesK + ln * T::kPitchV + hl * 16;

  // one 64-key step over the LDS stage `cur`
  auto step = [&](const char* cur, int kb, auto masked) {
    constexpr bool kMasked = decltype(masked)::value;
    // S^T = K Q^T: two 32-key tiles
    f32x16 s[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const char* krow = cur + kt * 32 * T::kPitchK + klane;
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(krow + kk * 32);
        if (kk == 0) {
          const f32x16 zero = {};
          s[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[0], zero, 0, 0, 0);
        } else {
          s[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], s[kt], 0, 0, 0);
        }
      }
    }
    // lane (hl, ln), register i of tile kt holds key kb + kt*32 + (i/8)*16 + hl*8 + i%8
    if constexpr (kMasked) {
      const int lim = pos - kb - hl * 8;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          s[kt][i] = (kt * 32 + (i >> 3) * 16 + (i & 7)) <= lim ? s[kt][i] : -__builtin_inff();
    }
    float mx = fmaxf(s[0][0], s[0][1]);
#pragma unroll
    for (int i = 2; i < 16; ++i) mx = fmaxf(mx, s[0][i]);
#pragma unroll
    for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[1][i]);
    const float m_blk = pair_max(mx) * c;
    const bool grow = m_blk > m_ref + kRescaleLog2;
    if (__any(grow)) {  // wave-uniform
      const float alpha = grow ? __builtin_amdgcn_exp2f(m_ref - m_blk) : 1.0f;
      m_ref = grow ? m_blk : m_ref;
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt) oacc[dt] *= alpha;
    }
    // a row with no visible key so far keeps m_ref = -inf; its scores are -inf too
    const float nm = m_ref == -__builtin_inff() ? 0.0f : -m_ref;
    uint32_t pk[2][8];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int i = 0; i < 16; i += 2)
        pk[kt][i >> 1] = pack_bf16x2(__builtin_amdgcn_exp2f(__builtin_fmaf(s[kt][i], c, nm)),
                                     __builtin_amdgcn_exp2f(__builtin_fmaf(s[kt][i + 1], c, nm)));
    // the row sum adds the same bf16-rounded weights that enter the PV
    // product, so the normalised weights sum to one exactly
    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
    float ls = 0.0f;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int j = 0; j < 8; ++j)
        ls = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pk[kt][j]), ones, ls, false);
    l_run += ls;
    // O^T += V^T P^T: 4 steps of 16 keys; step ks takes keys 16*ks + hl*8 .. +8
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const uint4 u = make_uint4(pk[ks >> 1][(ks & 1) * 4 + 0], pk[ks >> 1][(ks & 1) * 4 + 1],
                                 pk[ks >> 1][(ks & 1) * 4 + 2], pk[ks >> 1][(ks & 1) * 4 + 3]);
      const bf16x8 pb = __builtin_bit_cast(bf16x8, u);
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(cur + vlane + dt * 32 * T::kPitchV + ks * 32);
        oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb, oacc[dt], 0, 0, 0);
      }
    }
  };

  const int nsteps = (w.kv_hi - w.kv_lo + kKvStep - 1) / kKvStep;
  load(w.kv_lo);
  store(smem);
  __syncthreads();

  for (int it = 0; it < nsteps; ++it) {
    const int kb = w.kv_lo + it * kKvStep;
    const char* cur = smem + (it & 1) * T::kStage;
    char* nxt = smem + ((it + 1) & 1) * T::kStage;
    const bool more = it + 1 < nsteps;
    if (more) load(kb + kKvStep);
    if (kb <= pmax) {  // some row of this wave sees a key of this step
      if (kb + kKvStep - 1 > pmin)
        step(cur, kb, std::true_type{});
      else
        step(cur, kb, std::false_type{});
    }
    if (more) store(nxt);
    __syncthreads();
  }

  // epilogue: lane (hl, ln) holds row r, channels dt*32 + (i/4)*8 + hl*4 + i%4
  const float l_tot = pair_sum(l_run);
  if (!valid) return;
  if (w.out_slot < 0) {
    const float inv = 1.0f / l_tot;
    uint16_t* orow = p.o + (int64_t)tok * p.o_st + (int64_t)head * p.o_sh;
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const uint2 v = make_uint2(pack_bf16x2(oacc[dt][g4 * 4 + 0] * inv, oacc[dt][g4 * 4 + 1] * inv),
                                   pack_bf16x2(oacc[dt][g4 * 4 + 2] * inv, oacc[dt][g4 * 4 + 3] * inv));
        *reinterpret_cast<uint2*>(orow + dt * 32 + g4 * 8 + hl * 4) = v;
      }
    if (p.lse && hl == 0)
      p.lse[(int64_t)tok * p.num_q_heads + head] = (m_ref + __log2f(l_tot)) * kLn2;
  } else {
    float* slot = p.ws + (int64_t)w.out_slot * kRows * (D + 1);
    const bool empty = !(l_tot > 0.0f);  // no visible key in this split
    const float inv = empty ? 0.0f : 1.0f / l_tot;
    float* orow = slot + r * D;
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        f32x4 v;
#pragma unroll
        for (int j = 0; j < 4; ++j) v[j] = oacc[dt][g4 * 4 + j] * inv;
        *reinterpret_cast<f32x4*>(orow + dt * 32 + g4 * 8 + hl * 4) = v;
      }
    if (hl == 0)
      slot[kRows * D + r] = empty ? -__builtin_inff() : (m_ref + __log2f(l_tot)) * kLn2;
  }
}

template <int D>
__global__ __launch_bounds__(256) void msa_merge_kernel(MergeParams p) {
  constexpr int kThreadsPerRow = D / 4;
  constexpr int kRowsPerPass = 256 / kThreadsPerRow;
  const MergeItem mi = p.merge[blockIdx.x];
  const int G = p.group;
  const int rows = mi.nrows * G;
  const int sub = threadIdx.x % kThreadsPerRow;
  const int R = p.tile_rows;
  const int64_t slot_f = (int64_t)R * (D + 1);
  for (int r = threadIdx.x / kThreadsPerRow; r < rows; r += kRowsPerPass) {
    const int t = r / G, hh = r - t * G;
    const int tok = mi.row0 + t, head = mi.kv_head * G + hh;
    float mx = -__builtin_inff();
    for (int s = 0; s < mi.nsplit; ++s)
      mx = fmaxf(mx, p.ws[(int64_t)(mi.slot0 + s) * slot_f + (int64_t)R * D + r]);
    const float mu = mx == -__builtin_inff() ? 0.0f : mx;
    float L = 0.0f;
    f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int s = 0; s < mi.nsplit; ++s) {
      const float* base = p.ws + (int64_t)(mi.slot0 + s) * slot_f;
      const float wgt = __builtin_amdgcn_exp2f((base[(int64_t)R * D + r] - mu) * kLog2e);
      L += wgt;
      const f32x4 os = *reinterpret_cast<const f32x4*>(base + r * D + sub * 4);
      acc += wgt * os;
    }
    const float inv = L > 0.0f ? 1.0f / L : 0.0f;
    bf16x4 v;
#pragma unroll
    for (int j = 0; j < 4; ++j) v[j] = (__bf16)(acc[j] * inv);
    *reinterpret_cast<bf16x4*>(p.o + (int64_t)tok * p.o_st + (int64_t)head * p.o_sh + sub * 4) = v;
    if (p.lse && sub == 0) p.lse[(int64_t)tok * p.num_q_heads + head] = mu + __logf(L);
  }
}

}  // namespace

int launch_attn(const AttnParams& p, int head_dim, int tile_rows, int num_work, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (num_work <= 0) return 0;
  if (head_dim == 128 && tile_rows == kTileRowsNarrow)
    hipLaunchKernelGGL((msa_attn_kernel<128, 4>), dim3(num_work), dim3(256), 0, s, p);
  else if (head_dim == 128 && tile_rows == kTileRowsWide)
    hipLaunchKernelGGL((msa_attn_kernel<128, 8>), dim3(num_work), dim3(512), 0, s, p);
  else if (head_dim == 64 && tile_rows == kTileRowsNarrow)
    hipLaunchKernelGGL((msa_attn_kernel<64, 4>), dim3(num_work), dim3(256), 0, s, p);
  else if (head_dim == 64 && tile_rows == kTileRowsWide)
    hipLaunchKernelGGL((msa_attn_kernel<64, 8>), dim3(num_work), dim3(512), 0, s, p);
  else
    return (int)hipErrorInvalidValue;
  return (int)hipGetLastError();
}

int launch_merge(const MergeParams& p, int head_dim, int num_merge, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (num_merge <= 0) return 0;
  if (head_dim == 128)
    hipLaunchKernelGGL(msa_merge_kernel<128>, dim3(num_merge), dim3(256), 0, s, p);
  else if (head_dim == 64)
    hipLaunchKernelGGL(msa_merge_kernel<64>, dim3(num_merge), dim3(256), 0, s, p);
  else
    return (int)hipErrorInvalidValue;
  return (int)hipGetLastError();
}

}  // namespace msa
