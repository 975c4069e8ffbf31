// Host-side prefix metadata (radix tree of shared KV blocks) and the kernel
// work list. See tts_meta.h for the definitions.
#include "tts_meta.h"

#include <algorithm>
#include <cstdio>
#include <numeric>

namespace tts {
namespace {

constexpr int kErrInvalid = -1;
constexpr int kErrOutOfRange = -3;

struct Node {
  int32_t depth;
  int32_t nbeams;
  int32_t minbeam;
  int32_t first_child;
  int32_t next_sibling;
  int32_t block;
  int32_t seg;
  int32_t first_end;  // first beam whose full-block path ends here (-1: none)
};

std::string fmt(const char* f, long long a = 0, long long b = 0, long long c = 0) {
  char buf[256];
  std::snprintf(buf, sizeof(buf), f, a, b, c);
  return buf;
}

}  // namespace

int build_host_meta(const MetaInput& in, HostMeta* out, std::string* err) {
  const int32_t S = in.num_seqs;
  const int32_t bs = in.block_size;
  if (in.num_reqs < 0 || S < 0) {
    *err = "num_reqs and num_seqs must be >= 0";
    return kErrInvalid;
  }
  if (bs <= 0) {
    *err = "block_size must be > 0";
    return kErrInvalid;
  }
  if (in.max_blocks < 0 || in.num_blocks < 0) {
    *err = "max_blocks_per_seq and num_blocks must be >= 0";
    return kErrInvalid;
  }
  if (!in.req_seq_offsets) {
    *err = "req_seq_offsets is NULL";
    return kErrInvalid;
  }
  if (S > 0 && (!in.block_tables || !in.seq_lens)) {
    *err = "block_tables / seq_lens is NULL";
    return kErrInvalid;
  }
  if (in.req_seq_offsets[0] != 0 || in.req_seq_offsets[in.num_reqs] != S) {
    *err = fmt("req_seq_offsets must start at 0 and end at num_seqs (%lld)", S);
    return kErrInvalid;
  }
  for (int32_t r = 0; r < in.num_reqs; ++r) {
    if (in.req_seq_offsets[r + 1] < in.req_seq_offsets[r]) {
      *err = fmt("req_seq_offsets decreases at request %lld", r);
      return kErrInvalid;
    }
  }
  const int64_t mb = in.max_blocks;
  for (int32_t b = 0; b < S; ++b) {
    const int64_t L = in.seq_lens[b];
    if (L < 0 || L > mb * bs) {
      *err = fmt("seq_lens[%lld] = %lld outside [0, max_blocks_per_seq * block_size]", b, L);
      return kErrInvalid;
    }
    const int64_t nblk = (L + bs - 1) / bs;
    for (int64_t j = 0; j < nblk; ++j) {
      const int32_t id = in.block_tables[b * mb + j];
      if (id < 0 || id >= in.num_blocks) {
        *err = fmt("block_tables[%lld][%lld] = %lld outside [0, num_blocks)", b, j, id);
        return kErrOutOfRange;
      }
    }
  }

  HostMeta& m = *out;
  m = HostMeta();
  m.num_seqs = S;
  m.block_size = bs;
  m.max_blocks = in.max_blocks;
  m.tables.assign(in.block_tables, in.block_tables + static_cast<size_t>(S) * mb);
  m.seq_lens.assign(in.seq_lens, in.seq_lens + S);
  m.tail_lblock.assign(S, 0);
  m.req_off.assign(in.req_seq_offsets, in.req_seq_offsets + in.num_reqs + 1);
  m.perm.reserve(S);
  m.path_seg_off.assign(S + 1, 0);
  std::vector<std::vector<int32_t>> beam_segs(S);

  std::vector<Node> nodes;
  std::vector<int32_t> end_next(S, -1);
  std::vector<int32_t> path_nodes;      // per beam, CSR
  std::vector<int32_t> path_off(S + 1, 0);
  struct Item {
    int32_t key, kind, idx;  // kind 0: child node, 1: beam
  };
  std::vector<Item> items;
  std::vector<std::pair<int32_t, int32_t>> stack;  // (node or -(beam+1), parent node)

  for (int32_t r = 0; r < in.num_reqs; ++r) {
    const int32_t b0 = in.req_seq_offsets[r], b1 = in.req_seq_offsets[r + 1];
    if (b0 == b1) continue;
    nodes.clear();
    nodes.push_back(Node{0, 0, b0, -1, -1, -1, -1, -1});
    path_nodes.clear();
    // Insert each beam's full-block path, in original order.
    std::vector<int32_t> last_end(1, -1);
    for (int32_t b = b0; b < b1; ++b) {
      path_off[b - b0] = static_cast<int32_t>(path_nodes.size());
      int32_t cur = 0;
      nodes[0].nbeams++;
      const int32_t F = in.seq_lens[b] / bs;
      for (int32_t j = 0; j < F; ++j) {
        const int32_t id = in.block_tables[b * mb + j];
        int32_t c = nodes[cur].first_child;
        while (c >= 0 && nodes[c].block != id) c = nodes[c].next_sibling;
        if (c < 0) {
          c = static_cast<int32_t>(nodes.size());
          nodes.push_back(Node{nodes[cur].depth + 1, 0, b, -1, nodes[cur].first_child, id, -1, -1});
          nodes[cur].first_child = c;
        }
        nodes[c].nbeams++;
        cur = c;
        path_nodes.push_back(c);
      }
      // Append b to cur's list of ending beams, keeping ascending order.
      if (static_cast<int32_t>(last_end.size()) < static_cast<int32_t>(nodes.size()))
        last_end.resize(nodes.size(), -1);
      if (nodes[cur].first_end < 0) {
        nodes[cur].first_end = b;
      } else {
        end_next[last_end[cur]] = b;
      }
      last_end[cur] = b;
      end_next[b] = -1;
    }
    path_off[b1 - b0] = static_cast<int32_t>(path_nodes.size());

    // Depth-first walk; items at a node sorted by smallest original beam index.
    stack.clear();
    stack.emplace_back(0, -1);
    while (!stack.empty()) {
      auto [x, parent] = stack.back();
      stack.pop_back();
      if (x < 0) {
        m.perm.push_back(-x - 1);
        continue;
      }
      Node& nd = nodes[x];
      if (x != 0 && nd.nbeams >= 2) {
        if (parent != 0 && nodes[parent].nbeams == nd.nbeams) {
          nd.seg = nodes[parent].seg;
          m.seg_nblocks[nd.seg]++;
        } else {
          nd.seg = static_cast<int32_t>(m.seg_req.size());
          m.seg_req.push_back(r);
          m.seg_parent.push_back(parent != 0 ? nodes[parent].seg : -1);
          m.seg_lblock_begin.push_back(nd.depth - 1);
          m.seg_nblocks.push_back(1);
          m.seg_beam_begin.push_back(static_cast<int32_t>(m.perm.size()));
          m.seg_beam_end.push_back(static_cast<int32_t>(m.perm.size()) + nd.nbeams);
        }
      }
      items.clear();
      for (int32_t c = nd.first_child; c >= 0; c = nodes[c].next_sibling) items.push_back({nodes[c].minbeam, 0, c});
      for (int32_t b = nd.first_end; b >= 0; b = end_next[b]) items.push_back({b, 1, b});
      std::sort(items.begin(), items.end(), [](const Item& a, const Item& b) { return a.key < b.key; });
      for (auto it = items.rbegin(); it != items.rend(); ++it) {
        if (it->kind == 1)
          stack.emplace_back(-(it->idx + 1), -1);
        else
          stack.emplace_back(it->idx, x);
      }
    }
    // Tails and the covering segment of every shared block of each beam.
    for (int32_t b = b0; b < b1; ++b) {
      auto& segs = beam_segs[b];
      for (int32_t k = path_off[b - b0]; k < path_off[b - b0 + 1]; ++k) {
        const Node& nd = nodes[path_nodes[k]];
        if (nd.nbeams < 2) break;
        segs.push_back(nd.seg);
      }
      m.tail_lblock[b] = static_cast<int32_t>(segs.size());
    }
  }

  for (int32_t b = 0; b < S; ++b) m.path_seg_off[b + 1] = m.path_seg_off[b] + static_cast<int32_t>(beam_segs[b].size());
  m.path_seg.reserve(m.path_seg_off[S]);
  for (int32_t b = 0; b < S; ++b) m.path_seg.insert(m.path_seg.end(), beam_segs[b].begin(), beam_segs[b].end());
  m.pos_of.assign(S, 0);
  for (int32_t i = 0; i < S; ++i) m.pos_of[m.perm[i]] = i;

  // Unique physical blocks and tokens in use.
  std::vector<int32_t> best(static_cast<size_t>(in.num_blocks), 0);
  for (int32_t b = 0; b < S; ++b) {
    const int32_t L = in.seq_lens[b];
    const int32_t nblk = (L + bs - 1) / bs;
    for (int32_t j = 0; j < nblk; ++j) {
      const int32_t id = in.block_tables[b * mb + j];
      const int32_t v = std::min(bs, L - j * bs);
      if (best[id] == 0) m.unique_blocks++;
      if (v > best[id]) {
        m.unique_tokens += v - best[id];
        best[id] = v;
      }
    }
  }
  return 0;
}

int64_t coverage_rows(const HostMeta& m, const int32_t* seq_lens, int32_t* rows, int64_t cap) {
  const int32_t bs = m.block_size;
  int64_t n = 0;
  for (int32_t b = 0; b < m.num_seqs; ++b) {
    const int32_t L = seq_lens ? seq_lens[b] : m.seq_lens[b];
    const int32_t nblk = (L + bs - 1) / bs;
    const int32_t nseg = m.path_seg_off[b + 1] - m.path_seg_off[b];
    for (int32_t j = 0; j < nblk; ++j, ++n) {
      if (n >= cap) continue;
      int32_t* row = rows + n * 5;
      row[0] = b;
      row[1] = j;
      row[2] = j < m.max_blocks ? m.tables[static_cast<size_t>(b) * m.max_blocks + j] : -1;
      row[3] = std::min(bs, L - j * bs);
      row[4] = j < nseg ? m.path_seg[m.path_seg_off[b] + j] : -1;
    }
  }
  return n;
}


}  // namespace tts
