// Kernel work list of the prefix-shared decode attention.
//
// The attention kernel runs one persistent workgroup per compute unit; each
// workgroup walks a chain of unit records. A unit is a set of query rows
// (whole beams, consecutive in the canonical order, one KV head) and a list
// of KV blocks, each applying to a contiguous range of those rows. Two kinds
// of unit cover every (beam, used block) exactly once per KV head:
//
// * Wide units. A segment shared by more beams than fit in a narrow unit
//   (its rows exceed kMaxRows) is cut into row chunks of whole beams (up to
//   kMaxWideRows rows, or kAltWideRows where the cost model finds that plan
//   cheaper: the four waves of the workgroup share every block through
//   LDS, each taking a quarter of the row tiles) and, along its
//   blocks, into pieces; every (piece, chunk) is a unit whose blocks apply
//   to all of its rows. (fp32 caches use chunks of kMaxRows rows.) The
//   chunks of one piece read the same blocks and are placed on one XCD.
// * Narrow units. Everything else -- segments of few beams and every beam's
//   private tail -- is listed depth-first over the prefix tree (a segment's
//   blocks, then its subtrees and the tails of the beams ending at it, in
//   canonical order). Consecutive entries of that list always cover a
//   contiguous range of beams, so the list is cut into units of at most
//   kMaxUnitBeams beams / kMaxRows rows (kAltRows where the cost model
//   finds that plan cheaper) / kMaxEntries entries and about equal cost: a
//   small subtree with its tails becomes one unit and one partial state per
//   beam instead of one per segment.
//
// Units are replicated per KV head, grouped, spread over the XCDs longest
// first and then over each XCD's workgroups longest first.
#include <algorithm>
#include <cmath>
#include <numeric>

#include "tts_meta.h"

namespace tts {
namespace {

// Cost model (microseconds of one workgroup, all compute units busy),
// fitted to per-unit clock marks of the kernel at the 7B-shaped 64-beam
// tree (D 128, bf16 KV, g 7): every unit pays a fixed part (its first
// memory round trips, the end of its loop, the partial writes); a narrow
// unit then streams its blocks at about 0.21 us per 8 KiB block and pays
// about 0.08 us per query row (query read, combine, partial state); a wide
// unit pays about 0.193 us per 8 KiB block for staging it through LDS plus
// 0.113 us per block for each row tile a wave runs. (The narrow terms are
// the least-squares fit scaled by 1.25: a plain fit under-predicts the
// largest narrow units, which then finish last; the scale was chosen by
// timing the kernel.) fp32 caches scale the block terms by their bytes and
// every shape the tile term by the head size.
constexpr double kUnitFixedUs = 4.9;
constexpr double kNarrowUsPerByte = 0.2075 / 8192;
constexpr double kRowUs = 0.08;  // per row of 256 + 272 bytes (query + partial state)
constexpr double kWideUsPerByte = 0.193 / 8192;
constexpr double kTileBlockUs = 0.113;  // per block and row tile of a wave, D = 128
// fp8 caches: a block costs about what a bf16 block does (the products and
// the conversion, not the bytes, set its time), so they take their own
// terms, the least-squares fit to per-unit clock marks at the long-chain
// batch (16 x 32 beams, fp8 KV, 1,772 units): narrow 3.30 us + 0.204 us
// per block + 0.142 us per row, wide 4.60 us + 0.281 us per block + 0.093
// us per block and row tile of a wave.
constexpr double kFp8NarrowFixedUs = 3.30, kFp8NarrowBlockUs = 0.204, kFp8RowUs = 0.142;
constexpr double kFp8WideFixedUs = 4.60, kFp8WideBlockUs = 0.281, kFp8TileBlockUs = 0.093;
// When the units outnumber the workgroups (chained plans, where nearly every
// compute unit streams private blocks from HBM the whole time) a narrow
// unit's blocks take longer than at the 7B 64-beam tree: at the straggler
// batch the clock marks put narrow units at 1.24x the model and wide ones at
// 1.07x. Chained plans scale the bf16 narrow block term by 1.3 (1.15 to 1.6
// were timed; 1.3 was the fastest).
constexpr double kChainedNarrowScale = 1.3;
constexpr int kXcds = 8;  // workgroup k of a launch runs on XCD k % 8
constexpr int kAltWideRows = 128;  // the other wide-unit row cap the planner tries
constexpr int kAltRows = 42;       // the other narrow-unit row cap (plans that fit the workgroups)
// The merge (a second launch): a fixed cost plus one round trip to memory
// per kMergeBatch partial states of the beam with the most.
constexpr double kMergeFixedUs = 3.2;
constexpr double kMergeBatchUs = 1.4;

int tiles_of(int rows) { return (rows + 15) / 16; }

struct CostModel {
  double blk_bytes, q_row_bytes, part_row_bytes, d_scale;
  bool fp8 = false;
  double narrow_scale = 1.0;  // kChainedNarrowScale in chained plans
  double row_us() const { return kRowUs * (q_row_bytes + part_row_bytes) / 528.0; }
  double narrow_fixed() const { return fp8 ? kFp8NarrowFixedUs : kUnitFixedUs; }
  double wide_fixed() const { return fp8 ? kFp8WideFixedUs : kUnitFixedUs; }
  // Narrow units: the waves split the block pairs, every wave runs every tile.
  double narrow_us(int blocks, int rows) const {
    if (fp8) return kFp8NarrowFixedUs + blocks * kFp8NarrowBlockUs + rows * kFp8RowUs;
    return kUnitFixedUs + narrow_scale * blocks * blk_bytes * kNarrowUsPerByte + rows * row_us();
  }
  // Wide units: every wave runs every pair on its quarter of the tiles.
  double wide_us(int blocks, int rows) const {
    const int tpw = (tiles_of(rows) + 3) / 4;
    if (fp8) return kFp8WideFixedUs + blocks * (kFp8WideBlockUs + tpw * kFp8TileBlockUs * d_scale);
    return kUnitFixedUs + blocks * (blk_bytes * kWideUsPerByte + tpw * kTileBlockUs * d_scale);
  }
  // Bytes a unit moves: its blocks, its query rows, its partial states.
  double bytes(int blocks, int rows) const { return blocks * blk_bytes + rows * (q_row_bytes + part_row_bytes); }
};

struct Tmpl {
  int32_t lo = 0, hi = 0;  // beam positions [lo, hi)
  int32_t mode = kModeNarrow;
  std::vector<int32_t> ids;
  std::vector<uint32_t> info;
  int32_t nstatic = 0;   // narrow: static entries of the first window; wide: all entries
  int32_t nstatic2 = 0;  // narrow: entries of the second window (after the extension entries)
  double cost = 0;
  int32_t group = -1;  // wide units: index of their piece
};

struct NItem {
  int32_t id;
  int32_t p0, p1;
  int32_t valid;
  uint32_t flags;
};

struct Work {
  int32_t t, kvh;
  double cost;
};

// Which of a unit's beams (t.lo + i) it writes partial states for: all of
// a wide unit's; a narrow unit's whose rows some entry covers.
void touched_beams(const Tmpl& t, int32_t g, std::vector<char>* out) {
  const int32_t nb = t.hi - t.lo;
  out->assign(nb, t.mode == kModeWide ? 1 : 0);
  for (size_t k = 0; t.mode == kModeNarrow && k < t.ids.size(); ++k) {
    const uint32_t inf = t.info[k];
    const int32_t r0 = inf & 63, r1 = ((inf >> 6) & 63) + 1;
    for (int32_t i = r0 / g; i < (r1 + g - 1) / g && i < nb; ++i) (*out)[i] = 1;
  }
}

}  // namespace

void build_work_plan(const HostMeta& m, const PlanShape& shape, WorkPlan* plan, const WorkPlan* warm) {
  WorkPlan& P = *plan;
  P = WorkPlan();
  const int32_t S = m.num_seqs;
  const int32_t g = shape.num_q_heads / shape.num_kv_heads;
  const int32_t hkv = shape.num_kv_heads;
  const int32_t bs = m.block_size;
  // Beams per narrow unit: set per candidate row cap below.
  auto narrow_beams = [&](int32_t cap_rows) { return std::max(1, std::min(kMaxUnitBeams, cap_rows / g)); };
  int32_t RB = narrow_beams(kMaxRows);
  // Beams per wide unit (bf16 and fp8 caches; fp32 caches use narrow-sized
  // chunks): set per candidate row cap below.
  const bool wide_mode = shape.kv_bytes <= 2;
  int32_t RW = RB;
  auto wide_beams = [&](int32_t cap_rows) {
    return wide_mode ? std::max(1, std::min(kMaxWideBeams, cap_rows / g)) : RB;
  };
  const int32_t nseg = static_cast<int32_t>(m.seg_req.size());
  const int32_t nbins = std::max(1, shape.num_bins);
  P.num_bins = nbins;
  P.build_len.assign(m.seq_lens.begin(), m.seq_lens.end());

  CostModel cm;
  cm.blk_bytes = 2.0 * bs * shape.head_dim * shape.kv_bytes;
  cm.q_row_bytes = shape.head_dim * (shape.kv_bytes == 4 ? 4.0 : 2.0);
  // A partial state is written once and read once by the merge.
  cm.part_row_bytes = 2.0 * (shape.head_dim * (shape.kv_bytes == 4 ? 4.0 : 2.0) + 4 * kPartMl);
  cm.d_scale = shape.head_dim / 128.0;
  cm.fp8 = shape.kv_bytes == 1;

  // ---- tree structure ----------------------------------------------------
  std::vector<std::vector<int32_t>> children(nseg), leaves(nseg);
  std::vector<std::vector<std::pair<int32_t, int32_t>>> top(std::max<size_t>(1, m.req_off.size()) - 1);
  auto req_of_pos = [&](int32_t pos) {
    return static_cast<int32_t>(std::upper_bound(m.req_off.begin(), m.req_off.end(), pos) - m.req_off.begin()) - 1;
  };
  for (int32_t s = 0; s < nseg; ++s) {
    if (m.seg_parent[s] >= 0)
      children[m.seg_parent[s]].push_back(s);
    else
      top[m.seg_req[s]].push_back({m.seg_beam_begin[s], s});
  }
  for (int32_t pos = 0; pos < S; ++pos) {
    const int32_t b = m.perm[pos];
    const int32_t k0 = m.path_seg_off[b], k1 = m.path_seg_off[b + 1];
    if (k1 > k0)
      leaves[m.path_seg[k1 - 1]].push_back(pos);
    else
      top[req_of_pos(pos)].push_back({pos, -1 - pos});
  }
  std::vector<char> wide(nseg, 0);
  auto seg_block = [&](int32_t s, int32_t j) {
    const int32_t b = m.perm[m.seg_beam_begin[s]];
    return m.tables[static_cast<size_t>(b) * m.max_blocks + m.seg_lblock_begin[s] + j];
  };

  // ---- depth-first list of the narrow work --------------------------------
  std::vector<NItem> items;
  auto emit_tail = [&](int32_t pos) {
    const int32_t b = m.perm[pos];
    const int32_t L = m.seq_lens[b];
    const int32_t nb = (L + bs - 1) / bs;
    for (int32_t j = m.tail_lblock[b]; j < nb; ++j) {
      const int32_t v = std::min(bs, L - j * bs);
      const uint32_t fl = (j == nb - 1 && v < bs) ? kEntLive : 0u;
      items.push_back({m.tables[static_cast<size_t>(b) * m.max_blocks + j], pos, pos + 1, v, fl});
    }
    items.push_back({0, pos, pos + 1, 1, kEntExt});
  };
  // Iterative walk: a stack of (segment, or -1 - leaf position). Which
  // segments are wide (more beams than a narrow unit takes) depends on RB,
  // so the list is made again for each narrow row cap.
  std::vector<int32_t> stack;
  auto push_sorted = [&](std::vector<std::pair<int32_t, int32_t>>& v) {
    std::sort(v.begin(), v.end());
    for (auto it = v.rbegin(); it != v.rend(); ++it) stack.push_back(it->second);
  };
  std::vector<std::pair<int32_t, int32_t>> tmp;
  auto list_items = [&]() {
    for (int32_t s = 0; s < nseg; ++s) wide[s] = (m.seg_beam_end[s] - m.seg_beam_begin[s]) > RB;
    items.clear();
    for (auto& t : top) {
      push_sorted(t);
      while (!stack.empty()) {
        const int32_t x = stack.back();
        stack.pop_back();
        if (x < 0) {
          emit_tail(-1 - x);
          continue;
        }
        const int32_t bb = m.seg_beam_begin[x], be = m.seg_beam_end[x];
        if (!wide[x]) {
          for (int32_t j = 0; j < m.seg_nblocks[x]; ++j)
            items.push_back({seg_block(x, j), bb, be, bs, 0u});
        }
        tmp.clear();
        for (int32_t c : children[x]) tmp.push_back({m.seg_beam_begin[c], c});
        for (int32_t pos : leaves[x]) tmp.push_back({pos, -1 - pos});
        push_sorted(tmp);
      }
    }
  };

  // ---- units for a target unit time T ------------------------------------
  // A wide segment of G beams and n blocks is cut into C row chunks and P
  // pieces, in the wide mode (chunks of up to RW beams) or the narrow mode
  // (up to RB beams): the choice that moves the fewest bytes among those
  // whose units fit T (else the fastest). The narrow list is cut greedily
  // into units that fit T.
  auto make_templates = [&](double T, std::vector<Tmpl>& tm, int32_t& ngroups) {
    tm.clear();
    ngroups = 0;
    for (int32_t s = 0; s < nseg; ++s) {  // preorder: ancestors first
      if (!wide[s]) continue;
      const int32_t bb = m.seg_beam_begin[s], G = m.seg_beam_end[s] - bb;
      const int32_t n = m.seg_nblocks[s], np = (n + 1) / 2;
      struct Choice {
        int32_t mode, C, P;
        double bytes, us;
      } best{kModeNarrow, 0, 0, 0, 0};
      bool have = false, best_fits = false;
      for (int32_t mode : {kModeWide, kModeNarrow}) {
        if (mode == kModeWide && !wide_mode) continue;
        const int32_t cap = mode == kModeWide ? RW : RB;
        for (int32_t C = (G + cap - 1) / cap; C <= std::min(G, 4 * ((G + cap - 1) / cap)); ++C) {
          const int32_t rows = ((G + C - 1) / C) * g;
          const int32_t max_ent = mode == kModeWide ? kMaxUnitEntries : kMaxEntries;
          for (int32_t P = std::max(1, (n + max_ent - 1) / max_ent); P <= np; ++P) {
            const int32_t blocks = std::min(n, 2 * ((np + P - 1) / P));
            const double us = mode == kModeWide ? cm.wide_us(blocks, rows) : cm.narrow_us(blocks, rows);
            const double bytes = static_cast<double>(C) * P * cm.bytes(blocks, rows);
            const bool fits = us <= T;
            const bool better = !have || (fits && !best_fits) ||
                                (fits == best_fits && (fits ? bytes < best.bytes : us < best.us));
            if (better) {
              best = {mode, C, P, bytes, us};
              best_fits = fits;
              have = true;
            }
            if (fits) break;  // more pieces only add bytes
          }
        }
      }
      const int32_t C = best.C, pieces = best.P;
      for (int32_t j = 0; j < pieces; ++j) {
        const int32_t a = 2 * static_cast<int32_t>(static_cast<int64_t>(np) * j / pieces);
        const int32_t e = std::min(n, 2 * static_cast<int32_t>(static_cast<int64_t>(np) * (j + 1) / pieces));
        for (int32_t c = 0; c < C; ++c) {
          Tmpl t;
          t.lo = bb + static_cast<int32_t>(static_cast<int64_t>(G) * c / C);
          t.hi = bb + static_cast<int32_t>(static_cast<int64_t>(G) * (c + 1) / C);
          const int32_t rows = (t.hi - t.lo) * g;
          t.mode = best.mode;
          for (int32_t k = a; k < e; ++k) {
            t.ids.push_back(seg_block(s, k));
            t.info.push_back(t.mode == kModeWide ? 0u : ent_info(0, rows, bs, 0u));
          }
          t.nstatic = e - a;
          t.cost = t.mode == kModeWide ? cm.wide_us(e - a, rows) : cm.narrow_us(e - a, rows);
          t.group = ngroups;
          tm.push_back(std::move(t));
        }
        ++ngroups;
      }
    }
    Tmpl cur;
    std::vector<NItem> pend, ext;  // the open unit's static and extension items
    int32_t nblk = 0;
    // A unit's entries: the first window holds its LIVE entries, static
    // entries up to 64 with the extension entries, which come last; the
    // second window the remaining static entries (the order of a unit's
    // blocks does not change its result beyond rounding).
    auto flush = [&]() {
      if (pend.empty() && ext.empty()) return;
      auto push = [&](const NItem& it) {
        cur.ids.push_back(it.id);
        cur.info.push_back(ent_info((it.p0 - cur.lo) * g, (it.p1 - cur.lo) * g, it.valid, it.flags));
      };
      const int32_t room1 = kMaxEntries - static_cast<int32_t>(ext.size());
      int32_t nlive = 0;
      for (const NItem& it : pend) nlive += (it.flags & kEntLive) ? 1 : 0;
      int32_t plain1 = room1 - nlive;  // plain static entries the first window takes
      std::vector<const NItem*> second;
      for (const NItem& it : pend) {
        if ((it.flags & kEntLive) || plain1 > 0) {
          if (!(it.flags & kEntLive)) --plain1;
          push(it);
        } else {
          second.push_back(&it);
        }
      }
      cur.nstatic = static_cast<int32_t>(cur.ids.size());
      for (const NItem& it : ext) {
        cur.ids.push_back(it.p0 - cur.lo);
        cur.info.push_back(ent_info((it.p0 - cur.lo) * g, (it.p1 - cur.lo) * g, 1, kEntExt));
      }
      for (const NItem* it : second) push(*it);
      cur.nstatic2 = static_cast<int32_t>(second.size());
      cur.cost = cm.narrow_us(cur.nstatic + cur.nstatic2, (cur.hi - cur.lo) * g);
      tm.push_back(std::move(cur));
      cur = Tmpl();
      pend.clear();
      ext.clear();
      nblk = 0;
    };
    for (const NItem& it : items) {
      const bool is_ext = (it.flags & kEntExt) != 0;
      if (!pend.empty() || !ext.empty()) {
        const int32_t lo = std::min(cur.lo, it.p0), hi = std::max(cur.hi, it.p1);
        int32_t nlive = 0;
        for (const NItem& x : pend) nlive += (x.flags & kEntLive) ? 1 : 0;
        const int32_t live_ext = nlive + static_cast<int32_t>(ext.size()) +
                                 ((it.flags & (kEntLive | kEntExt)) ? 1 : 0);
        const bool fits = hi - lo <= RB && static_cast<int32_t>(pend.size() + ext.size()) + 1 <= kMaxUnitEntries &&
                          live_ext <= kMaxEntries && cm.narrow_us(nblk + (is_ext ? 0 : 1), (hi - lo) * g) <= T;
        if (!fits) flush();
      }
      if (pend.empty() && ext.empty()) {
        cur.lo = it.p0;
        cur.hi = it.p1;
      }
      cur.lo = std::min(cur.lo, it.p0);
      cur.hi = std::max(cur.hi, it.p1);
      if (is_ext) {
        ext.push_back(it);
      } else {
        pend.push_back(it);
        ++nblk;
      }
    }
    flush();
  };

  // ---- placement: groups -> XCDs -> workgroups ------------------------------
  // Units are replicated per KV head. The wide chunks of one piece (same
  // KV head) form a group that stays on one XCD, so they share its L2;
  // groups go to the XCDs longest first, then each XCD's units to its
  // workgroups longest first. Returns the largest workgroup load.
  auto place = [&](const std::vector<Tmpl>& tm, int32_t ngroups, std::vector<std::vector<Work>>& bins) {
    struct Group {
      double cost = 0;
      std::vector<Work> units;
    };
    std::vector<Group> groups;
    std::vector<int32_t> gidx(static_cast<size_t>(ngroups) * hkv, -1);
    for (int32_t kvh = 0; kvh < hkv; ++kvh) {
      for (size_t t = 0; t < tm.size(); ++t) {
        int32_t gi;
        if (tm[t].group >= 0) {
          int32_t& slot = gidx[static_cast<size_t>(tm[t].group) * hkv + kvh];
          if (slot < 0) {
            slot = static_cast<int32_t>(groups.size());
            groups.emplace_back();
          }
          gi = slot;
        } else {
          gi = static_cast<int32_t>(groups.size());
          groups.emplace_back();
        }
        groups[gi].units.push_back({static_cast<int32_t>(t), kvh, tm[t].cost});
        groups[gi].cost += tm[t].cost;
      }
    }
    std::vector<int32_t> gorder(groups.size());
    std::iota(gorder.begin(), gorder.end(), 0);
    std::stable_sort(gorder.begin(), gorder.end(),
                     [&](int32_t a, int32_t b) { return groups[a].cost > groups[b].cost; });
    const int32_t nx = std::min(kXcds, nbins);
    std::vector<int32_t> xbins(nx, 0);
    for (int32_t k = 0; k < nbins; ++k) xbins[k % nx]++;
    std::vector<double> xload(nx, 0);
    std::vector<std::vector<Work>> xunits(nx);
    for (int32_t gi : gorder) {
      int32_t x = 0;
      for (int32_t k = 1; k < nx; ++k)
        if (xload[k] / xbins[k] < xload[x] / xbins[x]) x = k;
      xload[x] += groups[gi].cost;
      for (const Work& w : groups[gi].units) xunits[x].push_back(w);
    }
    bins.assign(nbins, {});
    double makespan = 0;
    for (int32_t x = 0; x < nx; ++x) {
      auto& v = xunits[x];
      std::stable_sort(v.begin(), v.end(), [](const Work& a, const Work& b) { return a.cost > b.cost; });
      std::vector<int32_t> mine;
      for (int32_t k = x; k < nbins; k += nx) mine.push_back(k);
      std::vector<double> load(mine.size(), 0);
      for (const Work& w : v) {
        size_t best = 0;
        for (size_t k = 1; k < mine.size(); ++k)
          if (load[k] < load[best]) best = k;
        load[best] += w.cost;
        bins[mine[best]].push_back(w);
      }
      for (double l : load) makespan = std::max(makespan, l);
    }
    // Within a workgroup, wide units first (their chunks run concurrently on
    // the XCD's other workgroups and share its L2), then in creation order.
    for (auto& v : bins)
      std::stable_sort(v.begin(), v.end(), [](const Work& a, const Work& b) { return a.t < b.t; });
    return makespan;
  };

  // ---- target search ---------------------------------------------------------
  // Every unit pays a fixed cost and the kernel is bound by memory
  // bandwidth shared by all workgroups, so the best plan has one unit per
  // workgroup, all of about equal cost: the smallest target T whose units
  // (times the KV heads) still fit in the workgroups (a binary search; the
  // unit count only falls as T grows). When even the largest units
  // outnumber the workgroups, units are chained, and the target with the
  // smallest predicted makespan over a grid of candidates is taken.
  std::vector<Tmpl> tm;
  std::vector<std::vector<Work>> bins;
  int32_t ngroups = 0;
  const int32_t fit_units = std::max(1, nbins / hkv);
  auto units_at = [&](double T) {
    make_templates(T, tm, ngroups);
    return static_cast<int32_t>(tm.size());
  };
  // One search at the current RW: fills tm, bins, ngroups and the plan's
  // target, work and chaining; returns the modelled time it minimised (the
  // longest unit plus the merge for plans that fit the workgroups, the
  // largest workgroup load for chained ones).
  auto search = [&]() {
    cm.narrow_scale = 1.0;
    double est = 0;
    double work = 0;
    for (const NItem& it : items)
      if (!(it.flags & kEntExt)) work += cm.narrow_us(1, 0) - cm.narrow_fixed();
    for (int32_t s = 0; s < nseg; ++s)
      if (wide[s]) work += cm.wide_us(m.seg_nblocks[s], RW * g) - cm.wide_fixed();
    work = work * hkv / nbins;
    P.work_us = work;
    P.chained = false;
    if (warm && warm->target_us > 0 && warm->work_us > 0) {
      // Warm re-plan: the earlier target, scaled with the work, raised while
      // its units outnumber the workgroups (unless that plan was chained);
      // one placement, no search.
      double T = kUnitFixedUs + (warm->target_us - kUnitFixedUs) * (work / warm->work_us);
      T = std::max(T, kUnitFixedUs + 1e-3);
      if (!warm->chained)
        for (int it = 0; it < 12 && units_at(T) > fit_units; ++it) T = kUnitFixedUs + 1.15 * (T - kUnitFixedUs);
      units_at(T);
      est = place(tm, ngroups, bins);
      P.target_us = T;
      P.chained = warm->chained;
    } else {
      // Upper bound of the search: a few times the average work per unit,
      // raised while the units do not fit (one entry of many rows can cost
      // more than that bound by its row term alone; without the raise such a
      // batch would fall to the chained plans, with one tiny unit per entry).
      double hi = kUnitFixedUs + 4.0 * work + 1.0;
      for (int it = 0; it < 6 && units_at(hi) > fit_units; ++it) hi *= 2.0;
      if (units_at(hi) <= fit_units) {
        double lo = kUnitFixedUs;
        for (int it = 0; it < 24; ++it) {
          const double mid = 0.5 * (lo + hi);
          if (units_at(mid) <= fit_units)
            hi = mid;
          else
            lo = mid;
        }
        // Longer units mean fewer partial states per beam, so a cheaper merge:
        // take the target (the smallest one's variable part scaled up) with the
        // least modelled attention plus merge time.
        std::vector<char> touched;
        auto most_slots = [&](const std::vector<Tmpl>& t) {
          std::vector<int32_t> cnt(S, 0);
          for (const Tmpl& x : t) {
            touched_beams(x, g, &touched);
            for (int32_t i = 0; i < x.hi - x.lo; ++i)
              if (touched[i]) ++cnt[m.perm[x.lo + i]];
          }
          return S > 0 ? *std::max_element(cnt.begin(), cnt.end()) : 0;
        };
        const double t_min = hi;
        double best_T = t_min, best_est = -1;
        for (double f : {1.0, 1.5, 2.0, 3.0, 4.0, 6.0}) {
          const double T = kUnitFixedUs + f * (t_min - kUnitFixedUs);
          if (units_at(T) > fit_units) continue;
          double ms = 0;
          for (const Tmpl& x : tm) ms = std::max(ms, x.cost);
          const int32_t slots = most_slots(tm);
          const double est = ms + kMergeFixedUs + kMergeBatchUs * ((slots + kMergeBatch - 1) / kMergeBatch);
          if (best_est < 0 || est < best_est) {
            best_est = est;
            best_T = T;
          }
        }
        units_at(best_T);
        place(tm, ngroups, bins);
        P.target_us = best_T;
        est = best_est;
      } else {
        std::vector<Tmpl> cand;
        std::vector<std::vector<Work>> cbins;
        double best = -1;
        cm.narrow_scale = kChainedNarrowScale;
        for (double f : {0.35, 0.5, 0.65, 0.8, 1.0, 1.2, 1.45, 1.75, 2.1, 2.5, 3.0, 4.0}) {
          int32_t cg = 0;
          make_templates(kUnitFixedUs + f * work, cand, cg);
          const double ms = place(cand, cg, cbins);
          if (best < 0 || ms < best) {
            best = ms;
            tm.swap(cand);
            bins.swap(cbins);
            ngroups = cg;
            P.target_us = kUnitFixedUs + f * work;
          }
        }
        P.chained = true;
        est = best;
      }
    }
    return est;
  };

  // Row caps. Wide units of up to kMaxWideRows rows (three row tiles per
  // wave) or of up to kAltWideRows (two): fewer rows per chunk means more
  // chunks that stage the same blocks, but shorter units to balance. Then,
  // for plans that fit the workgroups, narrow units of up to kAltRows rows
  // instead of kMaxRows: more, shorter units. The model picks, comparing
  // plans of one kind only (both fit the workgroups, or both are chained);
  // a candidate must model strictly faster. Measured: 7B 64-beam tree 192 /
  // 64 rows; balanced tree and straggler batch 128-row wide units (-1.3 and
  // -1.7 us per call); 1.5B 16-beam tree 42-row narrow units (-1.5 us). A
  // warm re-plan keeps the earlier plan's caps.
  if (warm && warm->target_us > 0 && warm->work_us > 0) {
    P.wide_rows = warm->wide_rows > 0 ? warm->wide_rows : kMaxWideRows;
    P.narrow_rows = warm->narrow_rows > 0 ? warm->narrow_rows : kMaxRows;
    RB = narrow_beams(P.narrow_rows);
    RW = wide_beams(P.wide_rows);
    list_items();
    search();
  } else {
    P.wide_rows = kMaxWideRows;
    P.narrow_rows = kMaxRows;
    RW = wide_beams(kMaxWideRows);
    list_items();
    double best = search();
    // Runs the search at caps (wide, narrow) and keeps it if it models
    // faster than the plan at hand, else restores that plan.
    auto try_caps = [&](int32_t wide_rows, int32_t narrow_rows) {
      std::vector<Tmpl> tm0 = tm;
      std::vector<std::vector<Work>> bins0 = bins;
      const int32_t ngroups0 = ngroups, RW0 = RW, RB0 = RB;
      const double target0 = P.target_us, work0 = P.work_us;
      const bool chained0 = P.chained;
      RB = narrow_beams(narrow_rows);
      RW = wide_beams(wide_rows);
      if (RB != RB0) list_items();
      const double alt = search();
      if (P.chained == chained0 && alt < best) {
        best = alt;
        P.wide_rows = wide_rows;
        P.narrow_rows = narrow_rows;
        return;
      }
      RW = RW0;
      const bool relist = RB != RB0;
      RB = RB0;
      if (relist) list_items();
      tm.swap(tm0);
      bins.swap(bins0);
      ngroups = ngroups0;
      P.target_us = target0;
      P.work_us = work0;
      P.chained = chained0;
    };
    if (wide_mode && wide_beams(kAltWideRows) != RW) try_caps(kAltWideRows, P.narrow_rows);
    if (!P.chained && narrow_beams(kAltRows) != RB) try_caps(P.wide_rows, kAltRows);
  }

  // ---- partial rows and merge lists ----------------------------------------
  std::vector<int32_t> prow0(tm.size());
  std::vector<std::vector<int32_t>> per_beam(S);
  int32_t rows = 0;
  for (size_t t = 0; t < tm.size(); ++t) {
    prow0[t] = rows;
    const int32_t nb = tm[t].hi - tm[t].lo;
    std::vector<char> touched;
    touched_beams(tm[t], g, &touched);
    for (int32_t i = 0; i < nb; ++i)
      if (touched[i]) per_beam[m.perm[tm[t].lo + i]].push_back(rows + i * g);
    rows += nb * g;
  }
  P.rows_per_head = rows;
  P.slot_off.assign(S + 1, 0);
  for (int32_t b = 0; b < S; ++b) P.slot_off[b + 1] = P.slot_off[b] + static_cast<int32_t>(per_beam[b].size());
  P.slot_rows.reserve(P.slot_off[S]);
  for (int32_t b = 0; b < S; ++b) P.slot_rows.insert(P.slot_rows.end(), per_beam[b].begin(), per_beam[b].end());
  P.num_slots = static_cast<int64_t>(P.slot_rows.size());
  size_t most = 0;
  for (const auto& v : per_beam) most = std::max(most, v.size());
  P.slot_stride = std::max<int32_t>(kMergeBatch + 1, static_cast<int32_t>((most + 1 + 15) / 16 * 16));
  P.slot_tab.assign(static_cast<size_t>(S) * P.slot_stride, 0);
  for (int32_t b = 0; b < S; ++b) {
    int32_t* row = P.slot_tab.data() + static_cast<size_t>(b) * P.slot_stride;
    row[0] = static_cast<int32_t>(per_beam[b].size());
    std::copy(per_beam[b].begin(), per_beam[b].end(), row + 1);
  }

  // ---- records ---------------------------------------------------------------
  auto make_rec = [&](const Work& w) {
    UnitRec r{};
    const Tmpl& t = tm[w.t];
    r.kvh = w.kvh;
    r.nrows = (t.hi - t.lo) * g;
    r.nstatic = t.nstatic;
    r.nent = static_cast<int32_t>(t.ids.size());
    r.prow0 = prow0[w.t];
    r.next = -1;
    r.mode = t.mode;
    for (int32_t i = 0; i < t.hi - t.lo; ++i) r.beams[i] = m.perm[t.lo + i];
    // First window: entries [0, n1); second window: the rest.
    const size_t n1 = t.ids.size() - static_cast<size_t>(t.mode == kModeWide ? std::max(0, t.nstatic - kMaxEntries)
                                                                                : t.nstatic2);
    r.nstatic2 = static_cast<int32_t>(t.ids.size() - n1);
    if (t.mode == kModeNarrow) r.nent = static_cast<int32_t>(n1);
    if (r.nstatic2 > 0) P.two_windows = true;
    for (size_t k = 0; k < t.ids.size(); ++k) {
      if (k < n1) {
        r.ent_id[k] = t.ids[k];
        r.ent_info[k] = t.info[k];
      } else {
        r.ent_id2[k - n1] = t.ids[k];
        r.ent_info2[k - n1] = t.info[k];
      }
    }
    return r;
  };
  P.recs.assign(nbins, UnitRec{});
  for (int32_t k = 0; k < nbins; ++k) P.recs[k].next = -1;
  for (int32_t k = 0; k < nbins; ++k) {
    int32_t prev = -1;
    for (size_t i = 0; i < bins[k].size(); ++i) {
      int32_t idx;
      if (i == 0) {
        idx = k;
        P.recs[k] = make_rec(bins[k][i]);
      } else {
        idx = static_cast<int32_t>(P.recs.size());
        P.recs.push_back(make_rec(bins[k][i]));
      }
      if (prev >= 0) P.recs[prev].next = idx;
      prev = idx;
      P.num_units++;
    }
  }
}

}  // namespace tts
