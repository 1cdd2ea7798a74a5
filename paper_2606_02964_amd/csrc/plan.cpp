// plan.cpp -- host planner: segment descriptors -> per-row positions and the
// workgroup work list of one fused MSA launch.
//
// The paper dispatches every request segment to a group of CTAs inside a
// single kernel and gives each token its own "equivalent seq_len" through a
// precomputed array (Sec. 4.1).  Here:
//   1. rows: each packed query row gets its absolute position (its causal
//      limit is position + 1 keys);
//   2. tiles: consecutive rows of one sequence are packed into tiles of up to
//      tile_rows / G tokens (G = Hq / Hkv query heads share one KV head),
//      across segment gaps as long as the keys masked for the earlier rows
//      stay a small fraction of the tile's work.  tile_rows is 256 (one
//      workgroup per CU, each K/V step loaded once for 256 rows) when the
//      128-row tiling has many tiles and a long run of key steps per
//      workgroup slot, else 128 (two workgroups per CU: one's start-up and
//      tail overlap the other's work, and decode-heavy plans keep more key
//      streams in flight); it is 32 when no 128-row tile would hold more
//      than 32 rows (decode-like plans: the four waves of a workgroup then
//      split the tile's keys);
//   3. units: tile x KV head, keys [0, max position in tile + 1);
//   4. key splits: units longer than a third of a workgroup slot's share of
//      the work are cut into 64-aligned key ranges, merged later by
//      log-sum-exp; with 32-row tiles the cut length is the shortest whose
//      pieces all fit one round of the workgroup slots;
//   5. order: (sequence, KV head) groups are spread over the 8 XCDs (blockIdx
//      i runs on XCD i % 8) so tiles sharing K/V share one XCD's L2.  Inside
//      each XCD, groups start in decreasing order of their longest piece and
//      a group's pieces run back to back, longest first, so that no long
//      piece (a decode row over a long context) is left for the end;
//   6. workgroups: the launch is persistent, one workgroup per slot, each
//      with its own list of items; each XCD's queue is dealt out in order to
//      the least-loaded workgroup of that XCD.
#include "plan.h"

#include <algorithm>
#include <cmath>
#include <cstring>
#include <numeric>

namespace msa {
namespace {

constexpr int kXcds = 8;
constexpr int kCUs = 256;
constexpr int64_t kWideMinTiles = 1024;  // narrow tiles from which wide tiles pay
// 64-key steps per workgroup slot of the narrow tiling from which wide tiles
// pay: shorter plans gain more from two workgroups per CU (one's start-up
// and tail overlap the other's work) than from loading each K/V step once
// for 256 rows (measured crossover about 400 steps per slot)
constexpr double kWideMinStepsPerSlot = 384.0;
constexpr double kWasteFrac = 0.125;     // masked keys allowed per tile, relative
constexpr int64_t kMinSplitKeys = 1024;  // never split below this many keys

msa_status fail(std::string* err, msa_status st, const std::string& msg) {
  *err = msg;
  return st;
}

bool aligned8(int64_t x) { return x > 0 && (x % 8) == 0; }

struct Unit {
  int32_t seq, kv_head, row0, nrows, kv_hi;
};

}  // namespace

msa_status build_plan(const msa_shape* shape, const int32_t* seq_kv_len, const int32_t* seg_indptr,
                      const int32_t* seg_start, const int32_t* seg_len, const msa_plan_opts* opts,
                      HostPlan* out, std::string* err) {
  if (!shape || !out) return fail(err, MSA_ERR_INVALID_ARG, "shape and out must be non-null");
  const msa_shape& s = *shape;
  msa_plan_opts o{};
  if (opts) o = *opts;
  for (int i = 0; i < 5; ++i)
    if (o.reserved[i] != 0) return fail(err, MSA_ERR_INVALID_ARG, "opts.reserved must be zero");
  if (o.flags & ~(MSA_PLAN_HOST_ONLY | MSA_PLAN_NO_AUTO_SPLIT | MSA_PLAN_TILE_ROWS_128 |
                  MSA_PLAN_TILE_ROWS_256 | MSA_PLAN_TILE_ROWS_32 | MSA_PLAN_PRECISE_WEIGHTS))
    return fail(err, MSA_ERR_INVALID_ARG, "unknown opts.flags bits");
  {
    const int forced = !!(o.flags & MSA_PLAN_TILE_ROWS_128) + !!(o.flags & MSA_PLAN_TILE_ROWS_256) +
                       !!(o.flags & MSA_PLAN_TILE_ROWS_32);
    if (forced > 1)
      return fail(err, MSA_ERR_INVALID_ARG, "MSA_PLAN_TILE_ROWS_32, _128 and _256 are exclusive");
  }

  if (s.num_seqs < 0) return fail(err, MSA_ERR_INVALID_ARG, "num_seqs < 0");
  if (s.num_q_heads < 1 || s.num_kv_heads < 1)
    return fail(err, MSA_ERR_INVALID_ARG, "head counts must be >= 1");
  if (s.num_q_heads % s.num_kv_heads != 0)
    return fail(err, MSA_ERR_INVALID_ARG, "num_q_heads must be a multiple of num_kv_heads");
  const int32_t G = s.num_q_heads / s.num_kv_heads;
  if (G > kTileRowsWide) return fail(err, MSA_ERR_UNSUPPORTED, "num_q_heads / num_kv_heads > 256");
  if (G > kTileRowsNarrow && (o.flags & MSA_PLAN_TILE_ROWS_128))
    return fail(err, MSA_ERR_UNSUPPORTED, "128-row tiles need num_q_heads / num_kv_heads <= 128");
  if (G > kTileRowsDecode && (o.flags & MSA_PLAN_TILE_ROWS_32))
    return fail(err, MSA_ERR_UNSUPPORTED, "32-row tiles need num_q_heads / num_kv_heads <= 32");
  if (s.head_dim <= 0) return fail(err, MSA_ERR_INVALID_ARG, "head_dim <= 0");
  if (s.head_dim != 64 && s.head_dim != 128)
    return fail(err, MSA_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (s.block_size <= 0) return fail(err, MSA_ERR_INVALID_ARG, "block_size <= 0");
  if (s.block_size != kBlockSize) return fail(err, MSA_ERR_UNSUPPORTED, "block_size must be 16");
  if (s.max_blocks_per_seq < 0 || s.num_blocks < 0)
    return fail(err, MSA_ERR_INVALID_ARG, "max_blocks_per_seq and num_blocks must be >= 0");
  if (!std::isfinite(s.scale) || !(s.scale > 0.0f))
    return fail(err, MSA_ERR_INVALID_ARG, "scale must be finite and > 0");
  if (!aligned8(s.q_stride_tok) || !aligned8(s.q_stride_head) || !aligned8(s.o_stride_tok) ||
      !aligned8(s.o_stride_head) || !aligned8(s.k_stride_block) || !aligned8(s.k_stride_head) ||
      !aligned8(s.k_stride_tok) || !aligned8(s.v_stride_block) || !aligned8(s.v_stride_head) ||
      !aligned8(s.v_stride_dim))
    return fail(err, MSA_ERR_INVALID_ARG, "strides must be positive multiples of 8 elements");
  if (o.q_tile_tokens < 0 || o.q_tile_tokens > kTileRowsWide / G)
    return fail(err, MSA_ERR_INVALID_ARG, "q_tile_tokens must be in [0, tile_rows / (Hq/Hkv)]");
  if (o.kv_split_tokens < 0 || o.kv_split_tokens % kKvStep != 0)
    return fail(err, MSA_ERR_INVALID_ARG, "kv_split_tokens must be a non-negative multiple of 64");

  const int32_t B = s.num_seqs;
  if (B > 0 && (!seq_kv_len || !seg_indptr))
    return fail(err, MSA_ERR_INVALID_ARG, "seq_kv_len and seg_indptr must be non-null");
  if (B > 0 && seg_indptr[0] != 0) return fail(err, MSA_ERR_INVALID_ARG, "seg_indptr[0] != 0");
  for (int32_t b = 0; b < B; ++b)
    if (seg_indptr[b + 1] < seg_indptr[b])
      return fail(err, MSA_ERR_INVALID_ARG, "seg_indptr must be non-decreasing");
  const int64_t nseg = B > 0 ? seg_indptr[B] : 0;
  if (nseg > 0 && (!seg_start || !seg_len))
    return fail(err, MSA_ERR_INVALID_ARG, "seg_start and seg_len must be non-null");

  // 1. rows and their absolute positions
  HostPlan& P = *out;
  P = HostPlan{};
  P.shape = s;
  P.group = G;
  P.precise_weights = (o.flags & MSA_PLAN_PRECISE_WEIGHTS) != 0;
  std::vector<int64_t> seq_row0(B + 1, 0);
  std::vector<int32_t> seq_maxpos(B, -1);
  int64_t total = 0;
  const int64_t cap = (int64_t)s.max_blocks_per_seq * s.block_size;
  for (int32_t b = 0; b < B; ++b) {
    const int32_t L = seq_kv_len[b];
    if (L < 0 || L > cap)
      return fail(err, MSA_ERR_INVALID_ARG,
                  "seq_kv_len[" + std::to_string(b) + "] outside [0, max_blocks_per_seq*16]");
    int64_t prev_end = 0;
    seq_row0[b] = total;
    for (int32_t k = seg_indptr[b]; k < seg_indptr[b + 1]; ++k) {
      const int64_t st = seg_start[k], n = seg_len[k];
      if (n < 1) return fail(err, MSA_ERR_INVALID_ARG, "segment " + std::to_string(k) + " is empty");
      if (st < prev_end)
        return fail(err, MSA_ERR_INVALID_ARG,
                    "segment " + std::to_string(k) + " overlaps or is out of order");
      if (st + n > L)
        return fail(err, MSA_ERR_INVALID_ARG,
                    "segment " + std::to_string(k) + " extends past seq_kv_len");
      total += n;
      if (total >= ((int64_t)1 << 31)) return fail(err, MSA_ERR_INVALID_ARG, "total_q >= 2^31");
      prev_end = st + n;
      seq_maxpos[b] = (int32_t)(st + n - 1);
    }
  }
  seq_row0[B] = total;
  P.total_q = total;
  P.seq_blocks.resize((size_t)B);
  for (int32_t b = 0; b < B; ++b) P.seq_blocks[(size_t)b] = seq_maxpos[b] >= 0 ? seq_maxpos[b] / kBlockSize + 1 : 0;
  P.row_pos.resize((size_t)total);
  {
    int64_t r = 0;
    for (int32_t b = 0; b < B; ++b)
      for (int32_t k = seg_indptr[b]; k < seg_indptr[b + 1]; ++k)
        for (int32_t t = 0; t < seg_len[k]; ++t) P.row_pos[(size_t)r++] = seg_start[k] + t;
  }
  // 2. tiles of up to `tt` consecutive tokens of one sequence, packed
  // across segment gaps while the keys masked for the earlier rows stay a
  // small part of the tile's work; one unit per tile and KV head
  auto make_units = [&](int32_t tt) {
    std::vector<Unit> units;
    for (int32_t b = 0; b < B; ++b) {
      const int64_t lo = seq_row0[b], hi = seq_row0[b + 1];
      int64_t i = lo;
      while (i < hi) {
        const int64_t first = i;
        double useful = (double)P.row_pos[(size_t)i] + 1.0, waste = 0.0;
        int32_t cnt = 1;
        ++i;
        while (i < hi && cnt < tt) {
          const double step = (double)P.row_pos[(size_t)i] - (double)P.row_pos[(size_t)(i - 1)];
          const double nw = waste + cnt * step;
          const double nu = useful + (double)P.row_pos[(size_t)i] + 1.0;
          if (nw > kWasteFrac * nu && nw > (double)kKvStep * tt) break;
          waste = nw;
          useful = nu;
          ++cnt;
          ++i;
        }
        const int32_t kv_hi = P.row_pos[(size_t)(first + cnt - 1)] + 1;
        for (int32_t g = 0; g < s.num_kv_heads; ++g) units.push_back(Unit{b, g, (int32_t)first, cnt, kv_hi});
      }
    }
    return units;
  };

  // tile width: forced by a flag, else 32 rows when no 128-row tile would
  // hold more than 32 rows (decode-like plans), wide when the narrow tiling
  // has many tiles and enough work per workgroup slot (G > 128 needs wide
  // tiles), else narrow
  const int32_t narrow_tokens = G <= kTileRowsNarrow ? kTileRowsNarrow / G : 0;
  std::vector<Unit> narrow_units;
  {
    int32_t rows = kTileRowsNarrow;
    if (o.flags & MSA_PLAN_TILE_ROWS_256) {
      rows = kTileRowsWide;
    } else if (o.flags & MSA_PLAN_TILE_ROWS_32) {
      rows = kTileRowsDecode;
    } else if (!(o.flags & MSA_PLAN_TILE_ROWS_128)) {
      if (G > kTileRowsNarrow) {
        rows = kTileRowsWide;
      } else {
        narrow_units = make_units(narrow_tokens);
        double steps = 0;
        int64_t max_rows = 0;
        for (const Unit& u : narrow_units) {
          steps += (double)((u.kv_hi + kKvStep - 1) / kKvStep);
          max_rows = std::max<int64_t>(max_rows, (int64_t)u.nrows * G);
        }
        if (!narrow_units.empty() && max_rows <= kTileRowsDecode)
          rows = kTileRowsDecode;
        else if ((int64_t)narrow_units.size() >= kWideMinTiles && steps >= kWideMinStepsPerSlot * 2.0 * kCUs)
          rows = kTileRowsWide;
      }
    }
    P.tile_rows = rows;
    P.tile_tokens = rows / G;
    if (o.q_tile_tokens > P.tile_tokens)
      return fail(err, MSA_ERR_INVALID_ARG, "q_tile_tokens must be in [0, tile_rows / (Hq/Hkv)]");
    if (o.q_tile_tokens > 0) P.tile_tokens = o.q_tile_tokens;
  }
  const int32_t tile_tokens = P.tile_tokens;
  const int64_t slots_total = (int64_t)kCUs * (P.tile_rows == kTileRowsWide ? 1 : 2);

  // slices of the cache write: each segment cut at cache-block boundaries
  {
    int64_t r = 0;
    for (int32_t b = 0; b < B; ++b)
      for (int32_t k = seg_indptr[b]; k < seg_indptr[b + 1]; ++k) {
        int32_t p = seg_start[k];
        const int32_t end = seg_start[k] + seg_len[k];
        while (p < end) {
          const int32_t stop = std::min(end, (p / kBlockSize + 1) * kBlockSize);
          P.append.push_back(AppendItem{(int32_t)r, b, p, stop - p});
          r += stop - p;
          p = stop;
        }
      }
  }

  // 3. units of the chosen width
  std::vector<Unit> units = narrow_units.empty() || tile_tokens != narrow_tokens ? make_units(tile_tokens)
                                                                                : std::move(narrow_units);
  const int32_t Hkv = s.num_kv_heads, d = s.head_dim;
  P.num_tiles = (int64_t)units.size();

  // 4. key splits
  auto steps = [](int64_t keys) { return (keys + kKvStep - 1) / kKvStep; };
  int64_t split_keys = 0;  // 0: no split
  if (o.kv_split_tokens > 0) {
    split_keys = o.kv_split_tokens;
  } else if (!(o.flags & MSA_PLAN_NO_AUTO_SPLIT) && !units.empty()) {
    double total_steps = 0;
    for (const Unit& u : units) total_steps += (double)(steps(u.kv_hi) + 1);
    if (P.tile_rows == kTileRowsDecode) {
      // 32-row tiles (decode-like, bound by K/V streaming; the four waves of
      // a workgroup already split an item's keys): all pieces in one round
      // of the workgroup slots, the longest piece as short as possible, i.e.
      // the shortest 64-aligned piece length whose piece count fits the
      // slots (no split if the units alone exceed them)
      auto pieces_at = [&](int64_t len) {
        int64_t c = 0;
        for (const Unit& u : units) c += (u.kv_hi + len - 1) / len;
        return c;
      };
      int64_t longest = 0;
      for (const Unit& u : units) longest = std::max<int64_t>(longest, u.kv_hi);
      int64_t lo = kKvStep, hi = (longest + kKvStep - 1) / kKvStep * kKvStep;
      if ((int64_t)units.size() <= slots_total) {
        while (lo < hi) {  // smallest length with pieces_at(length) <= slots
          const int64_t mid = (lo / kKvStep + hi / kKvStep) / 2 * kKvStep;
          if (pieces_at(mid) <= slots_total) hi = mid; else lo = mid + kKvStep;
        }
        split_keys = std::max<int64_t>(kMinSplitKeys, lo);
      }
    } else {
      // aim at about 3 work items per workgroup slot: a unit longer than
      // this share of the total is cut into pieces no longer than the share
      const int64_t share = (int64_t)std::ceil(total_steps / (3.0 * slots_total)) * kKvStep;
      split_keys = std::max<int64_t>(kMinSplitKeys, share);
    }
  }
  struct Piece {
    int32_t unit, lo, hi, slot;
  };
  std::vector<Piece> pieces;
  int64_t slots = 0;
  for (size_t ui = 0; ui < units.size(); ++ui) {
    const Unit& u = units[ui];
    int64_t nsplit = 1;
    if (split_keys > 0) {
      if (u.kv_hi > split_keys)
        nsplit = (u.kv_hi + split_keys - 1) / split_keys;
    }
    if (nsplit <= 1) {
      pieces.push_back(Piece{(int32_t)ui, 0, u.kv_hi, -1});
      continue;
    }
    // equal 64-aligned chunks, last one takes the remainder
    int64_t chunk = ((u.kv_hi + nsplit - 1) / nsplit + kKvStep - 1) / kKvStep * kKvStep;
    nsplit = (u.kv_hi + chunk - 1) / chunk;
    const int32_t slot0 = (int32_t)slots;
    for (int64_t k = 0; k < nsplit; ++k) {
      const int64_t a = k * chunk, e = std::min<int64_t>(u.kv_hi, (k + 1) * chunk);
      pieces.push_back(Piece{(int32_t)ui, (int32_t)a, (int32_t)e, (int32_t)(slots++)});
    }
    P.merge.push_back(MergeItem{u.seq, u.kv_head, u.row0, u.nrows, (int32_t)nsplit, slot0, 0, 0});
    P.max_splits = std::max<int64_t>(P.max_splits, nsplit);
  }
  P.num_slots = slots;
  P.workspace_bytes = slots * slot_floats(d, P.tile_rows) * (int64_t)sizeof(float);

  // 5. order: groups (seq, kv head) -> XCD queues
  const int64_t ngroups = (int64_t)B * Hkv;
  std::vector<double> gcost((size_t)ngroups, 0.0);
  auto pcost = [&](const Piece& p) { return (double)(steps(p.hi - p.lo) + 1); };
  for (const Piece& p : pieces) {
    const Unit& u = units[(size_t)p.unit];
    gcost[(size_t)((int64_t)u.seq * Hkv + u.kv_head)] += pcost(p);
  }
  double total_cost = 0;
  for (double c : gcost) total_cost += c;
  std::vector<std::vector<int32_t>> queue(kXcds);
  std::vector<double> load(kXcds, 0.0);
  auto least_loaded = [&]() {
    return (int)(std::min_element(load.begin(), load.end()) - load.begin());
  };
  std::vector<int32_t> order(pieces.size());
  std::iota(order.begin(), order.end(), 0);
  // A group keeps one XCD unless it alone is a large part of an XCD's work
  // (few groups): then its pieces are spread by cost like independent work.
  std::vector<int64_t> gorder((size_t)ngroups);
  std::iota(gorder.begin(), gorder.end(), 0);
  std::stable_sort(gorder.begin(), gorder.end(),
                   [&](int64_t a, int64_t b) { return gcost[(size_t)a] > gcost[(size_t)b]; });
  std::vector<int32_t> ghome((size_t)ngroups, -1);
  const double big = 0.5 * total_cost / kXcds;
  for (int64_t gi : gorder) {
    if (gcost[(size_t)gi] <= 0 || gcost[(size_t)gi] > big) continue;
    const int x = least_loaded();
    ghome[(size_t)gi] = x;
    load[(size_t)x] += gcost[(size_t)gi];
  }
  // pieces in XCD-assignment order: by group cost (desc), then own cost (desc), then index
  std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) {
    const Unit& ua = units[(size_t)pieces[(size_t)a].unit];
    const Unit& ub = units[(size_t)pieces[(size_t)b].unit];
    const int64_t ga = (int64_t)ua.seq * Hkv + ua.kv_head, gb = (int64_t)ub.seq * Hkv + ub.kv_head;
    if (ga != gb && gcost[(size_t)ga] != gcost[(size_t)gb])
      return gcost[(size_t)ga] > gcost[(size_t)gb];
    if (ga != gb) return ga < gb;
    return pcost(pieces[(size_t)a]) > pcost(pieces[(size_t)b]);
  });
  for (int32_t pi : order) {
    const Unit& u = units[(size_t)pieces[(size_t)pi].unit];
    const int64_t gi = (int64_t)u.seq * Hkv + u.kv_head;
    int x = ghome[(size_t)gi];
    if (x < 0) {
      x = least_loaded();
      load[(size_t)x] += pcost(pieces[(size_t)pi]);
    }
    queue[(size_t)x].push_back(pi);
  }
  // 6. workgroups: one persistent workgroup per slot (256 for 256-row
  // tiles, one per CU; 512 otherwise, two per CU), or 8 per round of the
  // XCD queues when that is fewer.  Workgroup i runs on XCD i % 8 and works
  // through its own list of items, so no workgroup waits for a dispatch
  // between items.  Each XCD's pieces go, in queue order (below), to the
  // least-loaded workgroup of that XCD (cost: key steps plus one for the
  // per-item start-up), as a dynamic dispatch would hand them out; a
  // workgroup runs its list in that order.  A plan with at most one piece
  // per workgroup gets one each.
  size_t rounds = 0;
  for (const auto& q : queue) rounds = std::max(rounds, q.size());
  const int64_t nwg = std::min<int64_t>(slots_total, (int64_t)rounds * kXcds);
  std::vector<std::vector<int32_t>> wg_list((size_t)nwg);
  std::vector<double> wg_load((size_t)nwg, 0.0);
  // Inside each XCD the queue runs groups by decreasing longest piece (then
  // by id), a group's pieces adjacent and longest first, so that the
  // workgroups of an XCD work on the same groups at the same time and share
  // their K/V in that XCD's L2; ordering by total group cost alone would
  // leave a light group's long piece (a decode row over a long context) to
  // run last.
  std::vector<double> gmax((size_t)ngroups, 0.0);
  for (const Piece& p : pieces) {
    const Unit& u = units[(size_t)p.unit];
    double& m = gmax[(size_t)((int64_t)u.seq * Hkv + u.kv_head)];
    m = std::max(m, pcost(p));
  }
  for (int x = 0; x < kXcds; ++x) {
    auto& qx = queue[(size_t)x];
    std::stable_sort(qx.begin(), qx.end(), [&](int32_t a, int32_t b) {
      const Piece& pa = pieces[(size_t)a];
      const Piece& pb = pieces[(size_t)b];
      const Unit& ua = units[(size_t)pa.unit];
      const Unit& ub = units[(size_t)pb.unit];
      const int64_t ga = (int64_t)ua.seq * Hkv + ua.kv_head, gb = (int64_t)ub.seq * Hkv + ub.kv_head;
      if (gmax[(size_t)ga] != gmax[(size_t)gb]) return gmax[(size_t)ga] > gmax[(size_t)gb];
      if (ga != gb) return ga < gb;
      return pcost(pa) > pcost(pb);
    });
    for (int32_t pi : qx) {
      int64_t best = -1;
      for (int64_t wgi = x; wgi < nwg; wgi += kXcds)
        if (best < 0 || wg_load[(size_t)wgi] < wg_load[(size_t)best]) best = wgi;
      wg_list[(size_t)best].push_back(pi);
      wg_load[(size_t)best] += pcost(pieces[(size_t)pi]);
    }
  }
  // trailing workgroups with nothing to do are not launched
  int64_t launched = nwg;
  while (launched > 0 && wg_list[(size_t)launched - 1].empty()) --launched;
  P.wg_ptr.assign(1, 0);
  P.work.reserve(pieces.size());
  for (int64_t wgi = 0; wgi < launched; ++wgi) {
    for (int32_t pi : wg_list[(size_t)wgi]) {
      const Piece& p = pieces[(size_t)pi];
      const Unit& u = units[(size_t)p.unit];
      P.work.push_back(WorkItem{u.seq, u.kv_head, u.row0, u.nrows, p.lo, p.hi, p.slot, (int32_t)wgi});
    }
    P.wg_ptr.push_back((int32_t)P.work.size());
  }

  // figures
  const double hq = s.num_q_heads;
  for (int64_t r = 0; r < total; ++r) P.useful_flops += 4.0 * d * hq * ((double)P.row_pos[(size_t)r] + 1);
  const double qo_bytes = 2.0 * 2.0 * (double)total * hq * d;  // Q read + O write, bf16
  P.planned_bytes = qo_bytes;
  for (const WorkItem& w : P.work) {
    if (w.nrows == 0) continue;
    const double keys = (double)(w.kv_hi - w.kv_lo);
    P.planned_bytes += keys * d * 2.0 * 2.0;
    // waves whose 32 rows are all empty skip every step
    const double rows = (double)((w.nrows * G + 31) / 32 * 32);
    // 32-row tiles run 32-key half-steps, the others 64-key steps
    const int64_t gran = P.tile_rows == kTileRowsDecode ? kKvStep / 2 : kKvStep;
    P.tile_flops += 4.0 * d * rows * (double)((w.kv_hi - w.kv_lo + gran - 1) / gran * gran);
  }
  P.min_bytes = qo_bytes;
  for (int32_t b = 0; b < B; ++b)
    if (seq_maxpos[b] >= 0) P.min_bytes += (double)(seq_maxpos[b] + 1) * d * 2.0 * 2.0 * Hkv;
  return MSA_OK;
}

}  // namespace msa
