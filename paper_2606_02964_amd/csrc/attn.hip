// attn.hip -- gfx950 kernels of Multi-Segment Attention.
//
// msa_attn: workgroups of W waves (W = 4 or 8: 128 or 256 rows, 32 rows per
// wave), each running its own list of work items (the launch is persistent;
// the plan deals the items out).  A work item is query rows of one sequence
// sharing one KV head, over one key range.  Each 64-key step:
//   - paged gather: the step's 4 cache blocks are looked up in the block
//     table (ids preloaded one lane per step, read with v_readlane) and
//     copied straight into LDS (global_load_lds,
//     16 bytes a lane, no staging registers): K as [key][d] rows, V as the
//     cache's channel-major [d][16 keys] pages, 16-byte chunks XOR-swizzled
//     so that every operand read is free of bank conflicts.  K runs one step
//     ahead of V in rings of two stages.  The copies are inline assembly
//     (see dma16 for why);
//   - S^T = K Q^T on v_mfma_f32_32x32x16_bf16.  K is the A operand, so each
//     lane holds one query row (a column of S^T) and 16 of the 32 keys: the
//     row max and row sum need one exchange with the lane 32 apart only;
//   - per-row causal limit: key j is visible to the row at absolute position
//     p iff j <= p (only on steps that reach past the wave's smallest
//     position; a wave stops computing after the step holding its largest
//     position, while it keeps copying its share and meeting the barriers);
//   - online softmax in fp32 in the exp2 domain: scale * log2(e) enters one
//     FMA per score against a reference max that only moves (and O is only
//     rescaled) when a row's max grows by more than 2^8.  The row max itself
//     is only taken when a step's weights may have outgrown the reference
//     (see settle); the row sum adds the fp32 weights with plain adds (a
//     v_dot2 of the packed weights stalls the MFMA stream on gfx950);
//   - O^T += V^T P^T on the same MFMA, P packed to bf16 straight from the
//     score registers.  The A-operand row order of K is permuted (bits 2 and 3
//     of the row index swapped) so that the 8 scores a lane feeds to one PV
//     step are 8 consecutive keys, a single 16-byte LDS read of V^T.  On the
//     step holding a row's own position (its latest keys, and all keys of a
//     row near the start of a sequence) its weights enter as two bf16 terms,
//     hi = bf16(w) and lo = bf16(w - hi), with a second PV pass on lo, and
//     its row sum adds them in fp32: rows whose weight sits on a few keys
//     then carry their weights to about 2^-18 instead of 2^-9.
// Steps whose successor needs no mask run software-pipelined in pairs: the
// QK MFMAs of step j+1 are interleaved with the exponentials of step j, so
// that each of them is followed by independent vector work.  The diagonal
// steps and the last one run the same operations without overlap.
// msa_decode: 32-row tiles of decode-like plans; the four waves of a
// workgroup split the tile's keys, read K and V straight into registers and
// merge their softmax states through LDS (see the kernel); masked
// half-steps carry their weights as hi + lo terms, as above.
// Both kernels also come in a precise-weights form (kPrecise, selected by
// the plan): every step, or half-step, carries every row's weights as
// hi + lo terms, and the main kernel then runs every step unpipelined.
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

// LDS layout of one stage (no padding; 16-byte chunks XOR-swizzled so that
// every 16-lane group of an operand read hits 16 distinct bank groups):
//   K tile: 64 keys x D channels, row = key (2*D bytes); chunk c of row k is
//           stored at chunk c ^ ((k / rows per 256 bytes) mod chunks per row)
//   V tile: page-major, 4 blocks x D channels x 16 keys (32 bytes per channel
//           row); the two 16-byte halves of channel d swap when bit 3 of d is set
template <int D>
struct Tile {
  static constexpr int kBytesK = kKvStep * D * 2;
  static constexpr int kBytesV = kKvStep * D * 2;
  static constexpr int kPage = kBlockSize * D * 2;  // bytes of one block of K or V
  static constexpr int kDmaPerPage = kPage / 1024;  // 1 KB per wave-wide 16-byte copy
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

typedef __attribute__((address_space(3))) void lds_void_t;

// 16 bytes per lane from global memory (wave-uniform base + per-lane 32-bit
// byte offset) straight into LDS at lds + 16 * lane (a wave copies 1 KB; M0
// holds the wave's LDS base); completion is tracked by vmcnt.  The base goes
// in scalar registers, so the copy needs no vector address arithmetic.
// Issued as inline assembly: when the compiler sees these copies it treats
// the LDS counter as unordered and waits for every outstanding LDS read
// (lgkmcnt(0)) before each MFMA, which cancels the operand read-ahead.  The
// kernel itself waits for the copies (wait_dma) before the barrier that
// publishes them; the compiler's own vmcnt waits stay correct because vector
// loads complete in issue order, so extra loads it does not count only make
// those waits stricter.  The s_nop covers the M0-write-to-LDS-DMA hazard.
__device__ __forceinline__ void dma16(const void* base, uint32_t off, void* lds) {
  const uint32_t l = (uint32_t)(uintptr_t)(lds_void_t*)lds;
  asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(base), "{m0}"(l) : "memory");
}
// wait until at most n copies issued by this wave are outstanding
template <int n>
__device__ __forceinline__ void wait_dma() {
  static_assert(n >= 0 && n < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14));
}
// workgroup barrier that orders LDS accesses only: the compiler's
// __syncthreads() would also drain every outstanding global->LDS copy
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// running-max threshold of the lazy rescale: the reference max only moves
// when a row's max grows by more than this (log2 units), so the unnormalised
// weights stay <= 2^8
constexpr float kRescaleLog2 = 8.0f;
// a lane's step sum of weights at which the row max is taken (see settle)
constexpr float kSettleSum = 128.0f;

// One work item of msa_attn.  smem: the K ring (2 steps) then the V ring
// (2 steps).  Every wave leaves through the barrier that ends the item's
// last step before its epilogue (registers only), so the next item may
// refill the rings at once.
template <int D, int W, bool kPrecise>
__device__ __forceinline__ void attn_item(const AttnParams& p, const WorkItem w, char* smem) {
  using T = Tile<D>;
  constexpr int kRows = 32 * W;  // tile rows
  if (w.nrows == 0) return;  // (uniform over the workgroup)

  // lane-dependent set-up is computed per item (an opaque copy of the
  // thread id keeps it from being hoisted and held across items)
  int tid = threadIdx.x;
  asm volatile("" : "+v"(tid));
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int lane = tid & 63, hl = lane >> 5, ln = lane & 31;
  const int G = p.group;
  const int r = wave * 32 + ln;  // tile row
  const int t = r / G, hh = r - t * G;
  const bool valid = t < w.nrows;
  const int tok = w.row0 + t;
  const int head = w.kv_head * G + hh;
  const int pos = valid ? p.row_pos[tok] : -1;

  // wave-wide smallest and largest causal limit
  int pmin = valid ? pos : INT_MAX, pmax = pos;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    pmin = min(pmin, __shfl_xor(pmin, off));
    pmax = max(pmax, __shfl_xor(pmax, off));
  }
  pmin = __builtin_amdgcn_readfirstlane(pmin);
  pmax = __builtin_amdgcn_readfirstlane(pmax);

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

  // Gather geometry: a page (one block of K or V) is kDmaPerPage wave-wide
  // 16-byte copies (see the layout note above); lane offsets inside a block:
  constexpr int kChunksPerRow = 2 * D / 16;            // 16-byte chunks per K row
  constexpr int kRowsPerCopy = 64 / kChunksPerRow;     // K rows per 1 KB copy
  constexpr int kRowsPer256 = 256 / (2 * D);           // K rows sharing one 256-byte bank row
  auto kswz = [](int k) { return (k / kRowsPer256) & (kChunksPerRow - 1); };
  uint32_t kgo[T::kDmaPerPage];                       // byte offsets inside a cache block
#pragma unroll
  for (int q = 0; q < T::kDmaPerPage; ++q) {
    const int kin = q * kRowsPerCopy + lane / kChunksPerRow;
    const int lc = (lane % kChunksPerRow) ^ kswz(kin);
    kgo[q] = (uint32_t)(kin * p.k_st + lc * 8) * 2u;
  }
  // V copy q moves channels q*32 .. q*32+31: the same lane pattern, shifted
  // by 32 channels (bit 3 of the channel, hence the half swap, is unchanged)
  const uint32_t vgo0 = (uint32_t)((lane >> 1) * p.v_sd + (((lane & 1) ^ ((lane >> 4) & 1)) * 8)) * 2u;
  const uint32_t vgq = (uint32_t)(32 * p.v_sd) * 2u;
  const int64_t ksb = p.k_sb * 2, vsb = p.v_sb * 2;  // bytes per block
  const char* kbase = reinterpret_cast<const char*>(p.k + (int64_t)w.kv_head * p.k_sh);
  const char* vbase = reinterpret_cast<const char*>(p.v + (int64_t)w.kv_head * p.v_sh);
  const int32_t* bt = p.block_table + (int64_t)w.seq * p.max_blocks;
  auto kbuf = [&](int s) -> char* { return smem + __builtin_amdgcn_readfirstlane((s & 1) * T::kBytesK); };
  auto vbuf = [&](int s) -> char* {
    return smem + __builtin_amdgcn_readfirstlane(2 * T::kBytesK + (s & 1) * T::kBytesV);
  };
  const int n = (w.kv_hi - w.kv_lo + kKvStep - 1) / kKvStep;
  // A step has 8 pages: the K and the V page of each of its 4 blocks (page
  // pg: block pg & 3, V if pg >= 4); wave w copies pages w, w + W, ..., all
  // of block slot w & 3.  issue(sk, sv) copies the K pages of step sk and
  // the V pages of step sv (-1: none).  A block at or past kv_hi is not
  // read; its V page is zero-filled instead (its K page keeps old values:
  // those keys are masked by selection, so never meet arithmetic).
  // The block ids a wave needs sit in two registers, one lane per step:
  // lane i of idv0 holds the id of block slot w & 3 of step id_base + i, of
  // idv1 that of step id_base + 64 + i.  A step reads its id with
  // v_readlane (no memory access); every 64 steps the window moves on and
  // the next 64 ids load, 64 steps before they are needed.
  constexpr int kPagesPerWave = 8 / W;
  const int bslot = wave & 3;
  auto load_ids = [&](int s0) -> int32_t {
    const int st = s0 + lane;
    const int kb = w.kv_lo + st * kKvStep + bslot * kBlockSize;
    return (st < n && kb < w.kv_hi) ? bt[kb >> 4] : 0;
  };
  int id_base = 0;
  int32_t idv0 = load_ids(0), idv1 = load_ids(64);
  auto step_id = [&](int st) -> int64_t {  // id_base <= st < id_base + 128 (wave-uniform)
    const int i = st - id_base;
    return i < 64 ? __builtin_amdgcn_readlane(idv0, i) : __builtin_amdgcn_readlane(idv1, i - 64);
  };
  auto issue = [&](int sk, int sv) {
    if (sk >= id_base + 128) {  // move the window on (uniform; once per 64 steps)
      idv0 = idv1;
      idv1 = load_ids(id_base + 128);
      id_base += 64;
    }
    int64_t ids[kPagesPerWave];
    bool have[kPagesPerWave], zero[kPagesPerWave];
#pragma unroll
    for (int k = 0; k < kPagesPerWave; ++k) {
      const int pg = wave + k * W;
      const int bi = pg & 3;
      const int st = pg >= 4 ? sv : sk;
      const bool live = st >= 0 && st < n;
      const int kb = w.kv_lo + st * kKvStep;
      have[k] = live && kb + bi * kBlockSize < w.kv_hi;
      zero[k] = live && !have[k] && pg >= 4;
      ids[k] = have[k] ? step_id(st) : 0;
    }
#pragma unroll
    for (int k = 0; k < kPagesPerWave; ++k) {
      const int pg = wave + k * W;
      const int bi = pg & 3;
      if (have[k]) {
        if (pg < 4) {
          const char* kg = kbase + ids[k] * ksb;
          char* kd = kbuf(sk) + bi * T::kPage;
#pragma unroll
          for (int q = 0; q < T::kDmaPerPage; ++q) dma16(kg, kgo[q], kd + q * 1024);
        } else {
          const char* vg = vbase + ids[k] * vsb;
          char* vd = vbuf(sv) + bi * T::kPage;
#pragma unroll
          for (int q = 0; q < T::kDmaPerPage; ++q) dma16(vg + q * vgq, vgo0, vd + q * 1024);
        }
      } else if (zero[k]) {
#pragma unroll
        for (int q = 0; q < T::kDmaPerPage; ++q)
          *reinterpret_cast<uint4*>(vbuf(sv) + bi * T::kPage + q * 1024 + lane * 16) = make_uint4(0, 0, 0, 0);
      }
    }
  };

  const float c = p.scale_log2;  // > 0
  float m_ref = -__builtin_inff(), l_run = 0.0f;
  f32x16 oacc[D / 32];
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int i = 0; i < 16; ++i) oacc[dt][i] = 0.0f;
  const int krow_m = swap_bits23(ln);                 // key row of MFMA row ln (tile kt adds 32)
  const int vsw = (hl ^ ((ln >> 3) & 1)) * 16;        // V half swizzle of channel dt*32 + ln
  constexpr int kQk = 2 * (D / 16);                   // QK MFMAs per step, ordered (kk, kt)
  constexpr int kPv = 4 * (D / 32);                   // PV MFMAs per step, ordered (ks, dt)
  constexpr int kElPerQk = 32 / kQk;                  // scores handled per QK MFMA
  constexpr int kElPerPv = 32 / kPv;                  // scores handled per PV MFMA
  constexpr int kAhead = 3;                           // operand reads issued ahead of their MFMA

  // K operand of QK MFMA i of step s (register i of a lane: key row kt*32 + krow_m)
  auto kread_at = [&](const char* kb, int i) -> bf16x8 {
    const int kk = i >> 1, kt = i & 1;
    const int row = kt * 32 + krow_m;
    return *reinterpret_cast<const bf16x8*>(kb + row * (2 * D) + (((kk * 2 + hl) ^ kswz(row)) * 16));
  };
  auto vread_at = [&](const char* vb, int i) -> bf16x8 {
    const int ks = i / (D / 32), dt = i % (D / 32);
    return *reinterpret_cast<const bf16x8*>(vb + ks * T::kPage + (dt * 32 + ln) * 32 + vsw);
  };
  auto kread = [&](int s, int i) { return kread_at(kbuf(s), i); };
  auto vread = [&](int s, int i) { return vread_at(vbuf(s), i); };
  // the same with the ring stage known at compile time: its offset then
  // folds into the reads' immediate offsets
  auto kread_c = [&](auto st, int i) { return kread_at(smem + decltype(st)::value * T::kBytesK, i); };
  auto vread_c = [&](auto st, int i) {
    return vread_at(smem + 2 * T::kBytesK + decltype(st)::value * T::kBytesV, i);
  };
  // score e (0..31) of a lane sits in tile e/16, register e%16

  f32x16 sbuf[2][2];

  // QK of step s into sbuf[b] (no interleaving; prologue only)
  auto qk_plain = [&](int b, int s) {
#pragma unroll
    for (int i = 0; i < kQk; ++i) {
      const bf16x8 a = kread(s, i);
      const int kk = i >> 1, kt = i & 1;
      if (kk == 0) {
        const f32x16 zero = {};
        sbuf[b][kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[0], zero, 0, 0, 0);
      } else {
        sbuf[b][kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], sbuf[b][kt], 0, 0, 0);
      }
    }
  };
  // causal mask of step s applied to the scores in sbuf[b]
  auto mask_plain = [&](int b, int s) {
    const int lim = pos - (w.kv_lo + s * kKvStep) - hl * 8;
#pragma unroll
    for (int e = 0; e < 32; ++e) {
      const float x = sbuf[b][e >> 4][e & 15];
      sbuf[b][e >> 4][e & 15] = ((e >> 4) * 32 + ((e & 15) >> 3) * 16 + (e & 7)) <= lim ? x : -__builtin_inff();
    }
  };
  // weights of the scores in sbuf[b] against the reference max, packed to
  // bf16; ls gets the fp32 sum of the unrounded weights.  (The sum is taken
  // with plain adds: a v_dot2 of the packed weights against (1, 1) would be
  // one instruction per pair, but on gfx950 every dot2 stalls the matrix
  // core's MFMA stream for many cycles, while adds issue beside it.)
  auto weights_plain = [&](int b, uint32_t (&pk)[16], float& ls) {
    const float nm = m_ref == -__builtin_inff() ? 0.0f : -m_ref;
    ls = 0.0f;
#pragma unroll
    for (int e = 0; e < 32; e += 2) {
      const float w0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sbuf[b][e >> 4][e & 15], c, nm));
      const float w1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sbuf[b][(e + 1) >> 4][(e + 1) & 15], c, nm));
      pk[e >> 1] = pack_bf16x2(w0, w1);
      ls += w0 + w1;
    }
  };
  // On the step that holds a row's own position (its diagonal step) the
  // row's weights are carried as two bf16 terms: once the reference max is
  // settled, w replaces each score in sbuf[b] and the PV product runs on
  // hi = bf16(w) and on lo = bf16(w - hi)
  // (w - hi is exact in fp32), so hi + lo is within 2^-18 of w.  The
  // diagonal step holds a row's latest keys, and a row near the start of
  // the sequence has all its keys there: few keys then carry all the
  // weight, and a bf16 weight alone would move such a row's output by up to
  // about 2^-9 |v_i - v_j|.  Which steps do this depends on the row's own
  // position only (not on the rows sharing its wave), so a row's result
  // does not depend on its tile.
  auto weights_inplace = [&](int b) {
    const float nm = m_ref == -__builtin_inff() ? 0.0f : -m_ref;
#pragma unroll
    for (int e = 0; e < 32; ++e)
      sbuf[b][e >> 4][e & 15] = __builtin_amdgcn_exp2f(__builtin_fmaf(sbuf[b][e >> 4][e & 15], c, nm));
  };
  // packed bf16 lo terms of the weights e, e+1 held in sbuf[b], given their
  // hi terms (zero for a row off its diagonal step: own = false)
  auto lo_pair = [&](int b, int e, uint32_t hi, bool own) {
    const bf16x2 h = __builtin_bit_cast(bf16x2, hi);
    const uint32_t lo =
        pack_bf16x2(sbuf[b][e >> 4][e & 15] - (float)h[0], sbuf[b][(e + 1) >> 4][(e + 1) & 15] - (float)h[1]);
    return own ? lo : 0u;
  };
  // The row max is only taken when the weights of a step may have outgrown
  // the reference: a lane's step sum reached 2^7, or the row has no
  // reference yet.  A row whose max exceeds the reference by more than 2^8
  // (in log2 units) holds a weight >= 2^8, so its lane's sum passes 2^7:
  // the reference moves exactly as if the max were taken every step.  The
  // weights are then recomputed against the new reference.
  // (reweigh recomputes the step's weights and their sum ls.)
  auto settle = [&](int b, float ls, auto&& reweigh) {
    if (__any(!(ls < kSettleSum) || m_ref == -__builtin_inff())) {  // wave-uniform
      float mx = -__builtin_inff();
#pragma unroll
      for (int e = 0; e < 32; ++e) mx = fmaxf(mx, sbuf[b][e >> 4][e & 15]);
      const float m_blk = pair_max(mx) * c;
      const bool grow = m_blk > m_ref + kRescaleLog2;
      if (__any(grow)) {
        const float alpha = grow ? __builtin_amdgcn_exp2f(m_ref - m_blk) : 1.0f;
        m_ref = grow ? m_blk : m_ref;
        l_run *= alpha;
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt) oacc[dt] *= alpha;
        reweigh();
      }
    }
  };

  // One step j, scores of step j in sbuf[B] (masked):
  //   block 1: QK of step j+1 into sbuf[1-B], interleaved with the weights of
  //            step j; then settle the weights of step j (rarely does work)
  //   block 2: PV of step j (on diagonal steps interleaved with the mask of
  //            step j+1)
  // The source order is fixed with scheduling fences.  j has the parity of
  // B (the paired loop starts at step 0), so step j+1's K sits in ring stage
  // 1-B and step j's V in stage B.
  auto fused = [&](auto bsel, auto mask_next, auto has_next, int j) {
    constexpr int B = decltype(bsel)::value, NB = 1 - B;
    constexpr bool kMaskNext = decltype(mask_next)::value;
    constexpr bool kNext = decltype(has_next)::value;
    const float nm = m_ref == -__builtin_inff() ? 0.0f : -m_ref;
    uint32_t pk[16];
    float ls = 0.0f;
    // block 1
    bf16x8 ka[kQk];
    if constexpr (kNext) {
#pragma unroll
      for (int a = 0; a < kAhead; ++a) ka[a] = kread_c(std::integral_constant<int, NB>{}, a);
    }
#pragma unroll
    for (int i = 0; i < kQk; ++i) {
      if constexpr (kNext) {
        if (i + kAhead < kQk) ka[i + kAhead] = kread_c(std::integral_constant<int, NB>{}, i + kAhead);
        const int kk = i >> 1, kt = i & 1;
        if (kk == 0) {
          const f32x16 zero = {};
          sbuf[NB][kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[i], qf[0], zero, 0, 0, 0);
        } else {
          sbuf[NB][kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[i], qf[kk], sbuf[NB][kt], 0, 0, 0);
        }
      }
#pragma unroll
      for (int u = 0; u < kElPerQk; u += 2) {
        const int e = i * kElPerQk + u;
        const float w0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sbuf[B][e >> 4][e & 15], c, nm));
        const float w1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sbuf[B][(e + 1) >> 4][(e + 1) & 15], c, nm));
        pk[e >> 1] = pack_bf16x2(w0, w1);
        ls += w0 + w1;
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    settle(B, ls, [&]() { weights_plain(B, pk, ls); });
    l_run += ls;
    // block 2
    const int lim = pos - (w.kv_lo + (j + 1) * kKvStep) - hl * 8;
    bf16x8 va[kPv];
#pragma unroll
    for (int a = 0; a < kAhead; ++a) va[a] = vread_c(std::integral_constant<int, B>{}, a);
#pragma unroll
    for (int i = 0; i < kPv; ++i) {
      if (i + kAhead < kPv) va[i + kAhead] = vread_c(std::integral_constant<int, B>{}, i + kAhead);
      const int ks = i / (D / 32), dt = i % (D / 32);
      // P sub-step ks = keys 16*ks + hl*8 .. +8 = packed weights 4*ks .. 4*ks+3
      const bf16x8 pb = __builtin_bit_cast(bf16x8, make_uint4(pk[4 * ks], pk[4 * ks + 1], pk[4 * ks + 2], pk[4 * ks + 3]));
      oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[i], pb, oacc[dt], 0, 0, 0);
      if constexpr (kNext && kMaskNext) {
#pragma unroll
        for (int u = 0; u < kElPerPv; ++u) {
          const int e = i * kElPerPv + u;
          const float x = sbuf[NB][e >> 4][e & 15];
          sbuf[NB][e >> 4][e & 15] = ((e >> 4) * 32 + ((e & 15) >> 3) * 16 + (e & 7)) <= lim ? x : -__builtin_inff();
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // Step s's K sits in K buffer s % 2 and its V in V buffer s % 2; in
  // iteration j the copies of K_{j+2} and V_{j+1} are issued after the
  // barrier that ended iteration j-1 (the buffers' previous contents K_j and
  // V_{j-1} were last read before it) and waited for before the barrier that
  // ends iteration j.
  // (>=: a step whose last key is some row's position counts too, so that
  // every row's diagonal step runs through the masked path)
  auto need_mask = [&](int s) { return w.kv_lo + s * kKvStep + kKvStep - 1 >= pmin; };
  // steps this wave computes: keys up to its largest position.  A wave past
  // them still copies its share of every step and meets every barrier.
  const int nw = pmax >= w.kv_lo ? min(n, (pmax - w.kv_lo) / kKvStep + 1) : 0;
  issue(0, 0);
  issue(1, -1);
  wait_dma<0>();
  lds_barrier();
  if (nw > 0) {
    qk_plain(0, 0);
    if (need_mask(0)) mask_plain(0, 0);
  }
  lds_barrier();  // every wave is done with K_0 before K_2 replaces it

  // Iterations run in two loops.  The first handles two steps per trip
  // while both steps and their successors need no mask (the scores of step j
  // alternate between sbuf[0] and sbuf[1], so a trip starts and ends with
  // them in sbuf[0]).  The second handles the remaining steps (the diagonal
  // ones and the last) one at a time, copying the next scores back to
  // sbuf[0].  Waves may split their steps differently between the loops;
  // every step still ends with exactly one barrier.
  auto tail = [&]() {
    wait_dma<0>();
    lds_barrier();
  };
  // (with precise weights every step runs unpipelined, below)
  int j = 0;
  for (; !kPrecise && j + 2 < nw && !need_mask(j + 2); j += 2) {
    issue(j + 2, j + 1);
    fused(std::integral_constant<int, 0>{}, std::false_type{}, std::true_type{}, j);
    tail();
    issue(j + 3, j + 2);
    fused(std::integral_constant<int, 1>{}, std::false_type{}, std::true_type{}, j + 1);
    tail();
  }
  // Remaining steps (the diagonal ones and the last) run without overlap:
  // weights of step j, PV of step j, then QK + mask of step j+1 into the
  // same score registers.  Same copy schedule as the pipelined loop.
  // On a masked step (split: the diagonal step of some row of the wave) the
  // rows whose diagonal step it is also enter their weights' bf16 lo terms
  // (other rows: zeros), in a second PV pass after the usual one on pk.
  // With precise weights every step is split and every row enters them.
  auto plain = [&](int jj, bool split) {
    uint32_t pk[16];
    float ls;
    weights_plain(0, pk, ls);
    settle(0, ls, [&]() { weights_plain(0, pk, ls); });
    const int s_lo = w.kv_lo + jj * kKvStep;
    const bool own = pos >= s_lo && pos < s_lo + kKvStep;  // this is the row's diagonal step
    if (split) weights_inplace(0);  // the same weights in fp32, in place; hi(w) == pk
    l_run += ls;
#pragma unroll
    for (int i = 0; i < kPv; ++i) {
      const int ks = i / (D / 32), dt = i % (D / 32);
      const bf16x8 pb = __builtin_bit_cast(bf16x8, make_uint4(pk[4 * ks], pk[4 * ks + 1], pk[4 * ks + 2], pk[4 * ks + 3]));
      oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vread(jj, i), pb, oacc[dt], 0, 0, 0);
    }
    if (split) {
#pragma unroll
      for (int i = 0; i < kPv; ++i) {
        const int ks = i / (D / 32), dt = i % (D / 32);
        uint32_t pl[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) pl[u] = lo_pair(0, 8 * ks + 2 * u, pk[4 * ks + u], own || kPrecise);
        const bf16x8 pc = __builtin_bit_cast(bf16x8, make_uint4(pl[0], pl[1], pl[2], pl[3]));
        oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vread(jj, i), pc, oacc[dt], 0, 0, 0);
      }
    }
    if (jj + 1 < nw) {
      qk_plain(0, jj + 1);
      if (need_mask(jj + 1)) mask_plain(0, jj + 1);
    }
  };
  for (; j < n; ++j) {
    issue(j + 2, j + 1);
    if (j < nw) plain(j, kPrecise || need_mask(j));
    tail();
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
        for (int q = 0; q < 4; ++q) v[q] = oacc[dt][g4 * 4 + q] * inv;
        *reinterpret_cast<f32x4*>(orow + dt * 32 + g4 * 8 + hl * 4) = v;
      }
    if (hl == 0)
      slot[kRows * D + r] = empty ? -__builtin_inff() : (m_ref + __log2f(l_tot)) * kLn2;
  }
}

// Persistent launch: workgroup i runs the items wg_ptr[i] .. wg_ptr[i+1]-1.
template <int D, int W, bool kPrecise>
__global__ __launch_bounds__(64 * W, 2) void msa_attn_kernel(AttnParams p) {
  using T = Tile<D>;
  // K ring (2 steps) then V ring (2 steps); K runs one step ahead of V
  __shared__ __attribute__((aligned(1024))) char smem[2 * T::kBytesK + 2 * T::kBytesV];
  const int end = p.wg_ptr[blockIdx.x + 1];
  for (int it = p.wg_ptr[blockIdx.x]; it < end; ++it) attn_item<D, W, kPrecise>(p, p.work[it], smem);
}

// msa_decode: tiles of up to 32 rows (decode-like plans).  Every wave of the
// 4-wave workgroup holds the same 32 rows; wave w takes the 32-key
// half-steps w, w + 4, w + 8, ... of the item's key range and reads their K
// and V straight from the cache into MFMA operand registers.  A tile this
// small gains nothing from sharing K/V between waves through LDS, and
// registers hold more bytes in flight: each wave keeps the K of its next
// half-step and the V of its current one loading while it computes.  The
// four partial softmax states (max, sum, O) are merged through LDS at the
// end.  Arithmetic per half-step is that of the main kernel: S^T = K Q^T
// with K's rows permuted (bits 2 and 3 swapped), the lazy reference max,
// bf16 weights for the PV product and a row sum of the fp32 weights.
template <int D>
struct DecodeLds {
  static constexpr int kWaves = 4;
  static constexpr int kOPad = D + 4;  // row stride of the partial O (bank spread)
  float mo[kWaves][32][kOPad];
  float mm[kWaves][32], ml[kWaves][32];
};

// One work item of msa_decode; the LDS merge area is reused by the next item
// only after the barrier the caller places between items.
template <int D, bool kPrecise>
__device__ __forceinline__ void decode_item(const AttnParams& p, const WorkItem w, DecodeLds<D>& lds) {
  constexpr int kWaves = DecodeLds<D>::kWaves, kHalf = 32;
  auto& mo = lds.mo;
  auto& mm = lds.mm;
  auto& ml = lds.ml;
  if (w.nrows == 0) return;  // (uniform over the workgroup)

  // lane-dependent set-up is computed per item (an opaque copy of the
  // thread id keeps it from being hoisted and held across items)
  int tid = threadIdx.x;
  asm volatile("" : "+v"(tid));
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63, hl = lane >> 5, ln = lane & 31;
  const int G = p.group;
  const int t = ln / G, hh = ln - t * G;  // tile row ln <-> token t, head hh of the group
  const bool valid = t < w.nrows;
  const int tok = w.row0 + t;
  const int head = w.kv_head * G + hh;
  const int pos = valid ? p.row_pos[tok] : -1;
  int pmin = valid ? pos : INT_MAX, pmax = pos;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    pmin = min(pmin, __shfl_xor(pmin, off));
    pmax = max(pmax, __shfl_xor(pmax, off));
  }
  pmin = __builtin_amdgcn_readfirstlane(pmin);
  pmax = __builtin_amdgcn_readfirstlane(pmax);

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

  const char* kbase = reinterpret_cast<const char*>(p.k + (int64_t)w.kv_head * p.k_sh);
  const char* vbase = reinterpret_cast<const char*>(p.v + (int64_t)w.kv_head * p.v_sh);
  const int32_t* bt = p.block_table + (int64_t)w.seq * p.max_blocks;
  const int64_t ksb = p.k_sb * 2, vsb = p.v_sb * 2;  // bytes per block
  const int krow = swap_bits23(ln);                   // key (0..31 in the half-step) of MFMA row ln
  // per-lane byte offsets inside a block: K row krow % 16 at channel hl*8
  // (+ kk*16 per fragment); V^T row (channel) ln at keys hl*8 (+ dt*32 rows)
  const uint32_t koff = (uint32_t)((krow & 15) * p.k_st + hl * 8) * 2u;
  const uint32_t voff = (uint32_t)(ln * p.v_sd + hl * 8) * 2u;
  const uint32_t vdt = (uint32_t)(32 * p.v_sd) * 2u;

  const int nh = (w.kv_hi - w.kv_lo + kHalf - 1) / kHalf;
  // half-steps holding keys up to the tile's largest position
  const int nhw = pmax >= w.kv_lo ? min(nh, (pmax - w.kv_lo) / kHalf + 1) : 0;
  // The two blocks of half-step h.  The second one is only read when it
  // holds a key of the range; otherwise the first one stands in (its keys
  // are then past every row's position, hence masked).  The ids of this
  // wave's first 64 half-steps (h = wave + 4i) are loaded once, lane i
  // holding those of half-step i, so that no half-step waits for a table
  // read; later half-steps read the table directly.
  auto table_blocks = [&](int h, int32_t& id0, int32_t& id1) {
    const int k0 = w.kv_lo + h * kHalf;
    id0 = bt[k0 >> 4];
    id1 = k0 + kBlockSize < w.kv_hi ? bt[(k0 >> 4) + 1] : id0;
  };
  int32_t idv0 = 0, idv1 = 0;
  if (wave + kWaves * lane < nhw) table_blocks(wave + kWaves * lane, idv0, idv1);
  auto blocks = [&](int h, int64_t& id0, int64_t& id1) __attribute__((always_inline)) {
    const int i = (h - wave) / kWaves;  // wave-uniform
    if (i < 64) {
      id0 = __builtin_amdgcn_readlane(idv0, i);
      id1 = __builtin_amdgcn_readlane(idv1, i);
    } else {
      int32_t a, b;
      table_blocks(h, a, b);
      id0 = a;
      id1 = b;
    }
  };
  constexpr int kQk = D / 16;       // QK MFMAs per half-step
  constexpr int kPv = 2 * (D / 32); // PV MFMAs per half-step, ordered (ks, dt)
  bf16x8 ka[2][kQk], va[kPv];
  auto load_k = [&](auto bsel, int h) __attribute__((always_inline)) {
    constexpr int b = decltype(bsel)::value;
    int64_t id0, id1;
    blocks(h, id0, id1);
    const char* kb = kbase + (krow >= 16 ? id1 : id0) * ksb + koff;
#pragma unroll
    for (int kk = 0; kk < kQk; ++kk) ka[b][kk] = *reinterpret_cast<const bf16x8*>(kb + kk * 32);
  };
  auto load_v = [&](int h) __attribute__((always_inline)) {
    int64_t id0, id1;
    blocks(h, id0, id1);
#pragma unroll
    for (int i = 0; i < kPv; ++i) {
      const int ks = i / (D / 32), dt = i % (D / 32);
      va[i] = *reinterpret_cast<const bf16x8*>(vbase + (ks ? id1 : id0) * vsb + voff + dt * vdt);
    }
  };

  const float c = p.scale_log2;
  float m_ref = -__builtin_inff(), l_run = 0.0f;
  f32x16 oacc[D / 32];
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int i = 0; i < 16; ++i) oacc[dt][i] = 0.0f;

  // one half-step h of this wave, its K in buffer b
  auto half = [&](auto bsel, int h) __attribute__((always_inline)) {
    constexpr int b = decltype(bsel)::value;
    load_v(h);
    if (h + kWaves < nhw) load_k(std::integral_constant<int, 1 - b>{}, h + kWaves);
    f32x16 sc = {};
#pragma unroll
    for (int kk = 0; kk < kQk; ++kk) sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[b][kk], qf[kk], sc, 0, 0, 0);
    // score e (0..15) of a lane is key (e / 8) * 16 + hl * 8 + e % 8 of the half-step
    const int k0 = w.kv_lo + h * kHalf;
    // On a masked half-step (split) the rows whose diagonal half-step it is
    // also enter their weights' bf16 lo terms, as in the main kernel: a
    // second PV pass on them follows (with precise weights: on every
    // half-step, for every row).
    const bool masked = k0 + kHalf - 1 >= pmin;  // holds some row's position, or passes one
    const bool split = masked || kPrecise;
    if (masked) {
      const int lim = pos - k0 - hl * 8;
#pragma unroll
      for (int e = 0; e < 16; ++e) sc[e] = ((e >> 3) * 16 + (e & 7)) <= lim ? sc[e] : -__builtin_inff();
    }
    uint32_t pk[8];
    uint32_t plo[kPrecise ? 8 : 1];  // precise weights: the lo terms, taken with the hi ones
    float ls;
    auto weights = [&]() {
      const float nm = m_ref == -__builtin_inff() ? 0.0f : -m_ref;
      ls = 0.0f;
#pragma unroll
      for (int e = 0; e < 16; e += 2) {
        const float w0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[e], c, nm));
        const float w1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[e + 1], c, nm));
        pk[e >> 1] = pack_bf16x2(w0, w1);
        if constexpr (kPrecise) {
          const bf16x2 hv = __builtin_bit_cast(bf16x2, pk[e >> 1]);
          plo[e >> 1] = pack_bf16x2(w0 - (float)hv[0], w1 - (float)hv[1]);
        }
        ls += w0 + w1;  // fp32 sum (no v_dot2: it stalls the MFMA stream)
      }
    };
    weights();
    // the lazy reference max of the main kernel
    if (__any(!(ls < kSettleSum) || m_ref == -__builtin_inff())) {
      float mx = -__builtin_inff();
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = fmaxf(mx, sc[e]);
      const float m_blk = pair_max(mx) * c;
      const bool grow = m_blk > m_ref + kRescaleLog2;
      if (__any(grow)) {
        const float alpha = grow ? __builtin_amdgcn_exp2f(m_ref - m_blk) : 1.0f;
        m_ref = grow ? m_blk : m_ref;
        l_run *= alpha;
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt) oacc[dt] *= alpha;
        weights();
      }
    }
    const bool own = pos >= k0 && pos < k0 + kHalf;  // the row's diagonal half-step
    if (split && !kPrecise) {  // the same weights in fp32, in place of the scores; hi(w) == pk
      const float nm = m_ref == -__builtin_inff() ? 0.0f : -m_ref;
#pragma unroll
      for (int e = 0; e < 16; ++e) sc[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[e], c, nm));
    }
    l_run += ls;
#pragma unroll
    for (int i = 0; i < kPv; ++i) {
      const int ks = i / (D / 32), dt = i % (D / 32);
      const bf16x8 pb = __builtin_bit_cast(bf16x8, make_uint4(pk[4 * ks], pk[4 * ks + 1], pk[4 * ks + 2], pk[4 * ks + 3]));
      oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[i], pb, oacc[dt], 0, 0, 0);
    }
    if (split) {
#pragma unroll
      for (int i = 0; i < kPv; ++i) {
        const int ks = i / (D / 32), dt = i % (D / 32);
        uint32_t pl[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          if constexpr (kPrecise) {
            pl[u] = plo[4 * ks + u];
          } else {
            const bf16x2 hv = __builtin_bit_cast(bf16x2, pk[4 * ks + u]);
            pl[u] = own ? pack_bf16x2(sc[8 * ks + 2 * u] - (float)hv[0], sc[8 * ks + 2 * u + 1] - (float)hv[1]) : 0u;
          }
        }
        const bf16x8 pc = __builtin_bit_cast(bf16x8, make_uint4(pl[0], pl[1], pl[2], pl[3]));
        oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[i], pc, oacc[dt], 0, 0, 0);
      }
    }
  };
  if (wave < nhw) load_k(std::integral_constant<int, 0>{}, wave);
  for (int h = wave; h < nhw; h += 2 * kWaves) {
    half(std::integral_constant<int, 0>{}, h);
    if (h + kWaves < nhw) half(std::integral_constant<int, 1>{}, h + kWaves);
  }

  // merge the waves' partial states: lane (hl, ln) holds row ln, channels
  // dt*32 + (i/4)*8 + hl*4 + i%4
  const float l_tot = pair_sum(l_run);
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      f32x4 v;
#pragma unroll
      for (int q = 0; q < 4; ++q) v[q] = oacc[dt][g4 * 4 + q];
      *reinterpret_cast<f32x4*>(&mo[wave][ln][dt * 32 + g4 * 8 + hl * 4]) = v;
    }
  if (hl == 0) {
    mm[wave][ln] = m_ref;
    ml[wave][ln] = l_tot;
  }
  __syncthreads();
  constexpr int kCh = D / 8;  // channels per thread: 32 rows x 8 threads
  const int row = tid >> 3, c0 = (tid & 7) * kCh;
  const int rt = row / G, rh = row - rt * G;
  if (rt >= w.nrows) return;
  float M = -__builtin_inff();
#pragma unroll
  for (int u = 0; u < kWaves; ++u) M = fmaxf(M, mm[u][row]);
  float L = 0.0f, acc[kCh];
#pragma unroll
  for (int q = 0; q < kCh; ++q) acc[q] = 0.0f;
#pragma unroll
  for (int u = 0; u < kWaves; ++u) {
    const float f = mm[u][row] == -__builtin_inff() ? 0.0f : __builtin_amdgcn_exp2f(mm[u][row] - M);
    L += f * ml[u][row];
#pragma unroll
    for (int q = 0; q < kCh; q += 4) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(&mo[u][row][c0 + q]);
#pragma unroll
      for (int z = 0; z < 4; ++z) acc[q + z] += f * v[z];
    }
  }
  const int otok = w.row0 + rt, ohead = w.kv_head * G + rh;
  if (w.out_slot < 0) {
    const float inv = 1.0f / L;
    uint16_t* orow = p.o + (int64_t)otok * p.o_st + (int64_t)ohead * p.o_sh + c0;
#pragma unroll
    for (int q = 0; q < kCh; q += 4)
      *reinterpret_cast<uint2*>(orow + q) = make_uint2(pack_bf16x2(acc[q] * inv, acc[q + 1] * inv),
                                                       pack_bf16x2(acc[q + 2] * inv, acc[q + 3] * inv));
    if (p.lse && c0 == 0) p.lse[(int64_t)otok * p.num_q_heads + ohead] = (M + __log2f(L)) * kLn2;
  } else {
    constexpr int kR = 32;  // rows of a workspace slot of this tile width
    float* slot = p.ws + (int64_t)w.out_slot * kR * (D + 1);
    const bool empty = !(L > 0.0f);  // no visible key in this split
    const float inv = empty ? 0.0f : 1.0f / L;
#pragma unroll
    for (int q = 0; q < kCh; q += 4) {
      f32x4 v;
#pragma unroll
      for (int z = 0; z < 4; ++z) v[z] = acc[q + z] * inv;
      *reinterpret_cast<f32x4*>(slot + row * D + c0 + q) = v;
    }
    if (c0 == 0) slot[kR * D + row] = empty ? -__builtin_inff() : (M + __log2f(L)) * kLn2;
  }
}

template <int D, bool kPrecise>
__global__ __launch_bounds__(256, 2) void msa_decode_kernel(AttnParams p) {
  __shared__ __attribute__((aligned(16))) DecodeLds<D> lds;
  const int end = p.wg_ptr[blockIdx.x + 1];
  for (int it = p.wg_ptr[blockIdx.x]; it < end; ++it) {
    if (it > p.wg_ptr[blockIdx.x]) __syncthreads();  // the previous item's merge reads are done
    decode_item<D, kPrecise>(p, p.work[it], lds);
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

// The precise-weights forms are separate instantiations, so that the
// default kernels carry no test of the flag.
template <bool kPrecise>
int launch_attn_form(const AttnParams& p, int head_dim, int tile_rows, int num_wg, hipStream_t s) {
  if (head_dim == 128 && tile_rows == kTileRowsNarrow)
    hipLaunchKernelGGL((msa_attn_kernel<128, 4, kPrecise>), dim3(num_wg), dim3(256), 0, s, p);
  else if (head_dim == 128 && tile_rows == kTileRowsWide)
    hipLaunchKernelGGL((msa_attn_kernel<128, 8, kPrecise>), dim3(num_wg), dim3(512), 0, s, p);
  else if (head_dim == 64 && tile_rows == kTileRowsNarrow)
    hipLaunchKernelGGL((msa_attn_kernel<64, 4, kPrecise>), dim3(num_wg), dim3(256), 0, s, p);
  else if (head_dim == 64 && tile_rows == kTileRowsWide)
    hipLaunchKernelGGL((msa_attn_kernel<64, 8, kPrecise>), dim3(num_wg), dim3(512), 0, s, p);
  else if (head_dim == 128 && tile_rows == kTileRowsDecode)
    hipLaunchKernelGGL((msa_decode_kernel<128, kPrecise>), dim3(num_wg), dim3(256), 0, s, p);
  else if (head_dim == 64 && tile_rows == kTileRowsDecode)
    hipLaunchKernelGGL((msa_decode_kernel<64, kPrecise>), dim3(num_wg), dim3(256), 0, s, p);
  else
    return (int)hipErrorInvalidValue;
  return (int)hipGetLastError();
}

}  // namespace

int launch_attn(const AttnParams& p, int head_dim, int tile_rows, int num_wg, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (num_wg <= 0) return 0;
  return p.precise ? launch_attn_form<true>(p, head_dim, tile_rows, num_wg, s)
                   : launch_attn_form<false>(p, head_dim, tile_rows, num_wg, s);
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
