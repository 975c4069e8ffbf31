// Dynamic prefix-aware scheduling of reasoning paths (Sec. 4.2): order the
// active CoTs so that consecutive ones share long prefixes, then cut the
// order into batches that fit a KV memory budget. The eviction cost of a
// schedule is the sum over batches of the batch's trie size minus what it
// shares with the next batch.
#include <algorithm>
#include <cstdint>
#include <unordered_set>
#include <vector>

namespace tts {

struct SchedInput {
  int32_t num_cots;
  const int32_t* cot_off;    // [num_cots + 1]
  const int32_t* cot_nodes;  // node ids, root first
  const int64_t* weight;     // [num_nodes] or null (1 per node)
  int64_t budget;
};

struct SchedOutput {
  std::vector<int32_t> order, batch_off;
  int64_t score = 0, cost = 0;
};

static int32_t lcp(const SchedInput& in, int32_t a, int32_t b) {
  const int32_t* pa = in.cot_nodes + in.cot_off[a];
  const int32_t* pb = in.cot_nodes + in.cot_off[b];
  const int32_t n = std::min(in.cot_off[a + 1] - in.cot_off[a], in.cot_off[b + 1] - in.cot_off[b]);
  int32_t k = 0;
  while (k < n && pa[k] == pb[k]) ++k;
  return k;
}

// Greedy order: the first CoT, then repeatedly the remaining CoT sharing
// the longest prefix with the last one scheduled (ties: the earliest in the
// input, which keeps the relative order of the parents' groups).
// Batches: from the front, the longest run of consecutive CoTs whose trie
// (the union of their nodes) fits the budget; a CoT larger than the budget
// is a batch by itself.
void prefix_schedule(const SchedInput& in, SchedOutput* out) {
  const int32_t n = in.num_cots;
  out->order.clear();
  out->batch_off.assign(1, 0);
  out->score = out->cost = 0;
  if (n == 0) return;
  std::vector<char> used(n, 0);
  int32_t cur = 0;
  used[0] = 1;
  out->order.push_back(0);
  for (int32_t k = 1; k < n; ++k) {
    int32_t best = -1, best_l = -1;
    for (int32_t i = 0; i < n; ++i) {
      if (used[i]) continue;
      const int32_t l = lcp(in, cur, i);
      if (l > best_l) {
        best_l = l;
        best = i;
      }
    }
    used[best] = 1;
    out->score += best_l;
    out->order.push_back(best);
    cur = best;
  }
  auto w = [&](int32_t node) { return in.weight ? in.weight[node] : int64_t{1}; };
  // Batches, each with its node set; cost adds a batch's size minus the
  // weight of the nodes it shares with the next batch.
  std::unordered_set<int32_t> prev, open;
  int64_t open_size = 0;
  bool have_prev = false;
  int64_t prev_size = 0;
  auto close = [&]() {
    if (have_prev) {
      int64_t shared = 0;
      for (int32_t node : open)
        if (prev.count(node)) shared += w(node);
      out->cost += prev_size - shared;
    }
    prev.swap(open);
    open.clear();
    prev_size = open_size;
    open_size = 0;
    have_prev = true;
  };
  for (int32_t k = 0; k < n; ++k) {
    const int32_t c = out->order[k];
    int64_t add = 0;
    for (int32_t j = in.cot_off[c]; j < in.cot_off[c + 1]; ++j)
      if (!open.count(in.cot_nodes[j])) add += w(in.cot_nodes[j]);
    if (!open.empty() && open_size + add > in.budget) {
      out->batch_off.push_back(k);
      close();
      add = 0;
      for (int32_t j = in.cot_off[c]; j < in.cot_off[c + 1]; ++j)
        if (!open.count(in.cot_nodes[j])) add += w(in.cot_nodes[j]);
    }
    for (int32_t j = in.cot_off[c]; j < in.cot_off[c + 1]; ++j) open.insert(in.cot_nodes[j]);
    open_size += add;
  }
  out->batch_off.push_back(n);
  close();
  out->cost += prev_size;  // the last batch shares nothing with a successor
}

}  // namespace tts
