// Load-driven dynamic-CP scheduler (hydra_sched.h), heap-accelerated (Sec. 5.1.3).
//
// Per micro-batch the open groups live in one class per power-of-two size.  A class keeps
//   - a lazy min-heap of (load, start) entries: the least loaded group first, stale entries
//     (an older version of a group that has since taken a sequence) dropped when met;
//   - a max-heap of groups that failed the token test, keyed by remaining token capacity.
//     Sequences arrive longest first, so the per-rank token demand a class sees never grows:
//     a demoted group is re-admitted as soon as its capacity covers the current demand and
//     is otherwise never rescanned.
// A class whose least loaded group already sits at the target, with nothing demoted, is
// pruned until a new group of that size opens (loads only grow).  Free ranks are a bitset
// with one cursor per block size (blocks only ever become busy within a micro-batch), a
// min-heap by (size, start) drives backfill, and the maximum and minimum group loads for the
// balance test are kept incrementally.  Every choice uses the same keys and tie-breaks as a
// linear scan over the groups, so the placement is identical to it.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <functional>
#include <numeric>
#include <queue>
#include <vector>

#include "hydra_sched.h"

namespace hydra {
namespace {

typedef unsigned __int128 u128;

constexpr int64_t kMaxLen = int64_t(1) << 21;
constexpr int32_t kMaxRanks = 1 << 16;

int64_t ceil2_d(double x) {  // smallest power of two >= x
  int64_t p = 1;
  while ((double)p < x) p *= 2;
  return p;
}

struct Group {
  int32_t start, size;
  int64_t load, tokens;  // per rank, times C
  uint32_t ver;
};

struct LoadEntry {
  int64_t load;
  int32_t start, gid;
  uint32_t ver;
  bool operator>(const LoadEntry& o) const { return load != o.load ? load > o.load : start > o.start; }
};
struct CapEntry {
  int64_t remaining;
  int32_t start, gid;
  uint32_t ver;
  bool operator<(const CapEntry& o) const { return remaining != o.remaining ? remaining < o.remaining : start > o.start; }
};
struct SizeEntry {
  int32_t size, start, gid;
  bool operator>(const SizeEntry& o) const { return size != o.size ? size > o.size : start > o.start; }
};
struct MinLoad {
  int64_t load;
  int32_t gid;
  uint32_t ver;
  bool operator>(const MinLoad& o) const { return load > o.load; }
};

template <class T> using MinHeap = std::priority_queue<T, std::vector<T>, std::greater<T>>;

class FreeRanks {
 public:
  FreeRanks(int G, int levels) : G_(G), words_((G + 63) / 64), cursor_(levels + 1, 0) {}
  void reset() {
    used_.assign(words_, 0);
    std::fill(cursor_.begin(), cursor_.end(), 0);
    free_ = G_;
  }
  bool block_free(int32_t start, int32_t size) const {
    if (size < 64) {
      const uint64_t m = (size == 64 ? ~0ull : ((1ull << size) - 1)) << (start & 63);
      return (used_[start >> 6] & m) == 0;
    }
    for (int w = start >> 6; w < (start + size) >> 6; ++w)
      if (used_[w]) return false;
    return true;
  }
  void take(int32_t start, int32_t size) {
    if (size < 64) {
      used_[start >> 6] |= ((1ull << size) - 1) << (start & 63);
    } else {
      for (int w = start >> 6; w < (start + size) >> 6; ++w) used_[w] = ~0ull;
    }
    free_ -= size;
  }
  // lowest free block of `size` ranks aligned to `size` (level = log2 size), or -1
  int32_t lowest(int level) {
    const int32_t size = 1 << level;
    int32_t& c = cursor_[level];
    while ((int64_t)c * size < G_ && !block_free(c * size, size)) ++c;
    return (int64_t)c * size < G_ ? c * size : -1;
  }
  int free_count() const { return free_; }

 private:
  int G_, words_, free_ = 0;
  std::vector<uint64_t> used_;
  std::vector<int32_t> cursor_;
};

int log2i(int64_t p) {
  int l = 0;
  while ((int64_t(1) << l) < p) ++l;
  return l;
}

}  // namespace
}  // namespace hydra

extern "C" int hydra_schedule(const int64_t* lengths, int64_t n_docs, const hydra_sched_config_t* cfg, int32_t* mb,
                              int32_t* group_start, int32_t* group_size, hydra_sched_summary_t* summary) {
  using namespace hydra;
  if (!cfg || n_docs < 0 || (n_docs > 0 && (!lengths || !mb || !group_start || !group_size))) return HYDRA_ERR_INVALID;
  const int64_t G = cfg->n_ranks, B = cfg->token_budget;
  if (G < 1 || G > kMaxRanks || B < 1 || cfg->pp < 1) return HYDRA_ERR_INVALID;
  if (!(cfg->theta_over_c >= 0.0) || !std::isfinite(cfg->theta_over_c)) return HYDRA_ERR_INVALID;
  const double ratio = cfg->balance_ratio == 0.0 ? 0.9 : cfg->balance_ratio;
  if (!(ratio > 0.0 && ratio <= 1.0)) return HYDRA_ERR_INVALID;
  if (n_docs == 0) {
    if (summary) *summary = hydra_sched_summary_t{};
    return HYDRA_OK;
  }
  int64_t s_max = 0;
  u128 W = 0;
  for (int64_t i = 0; i < n_docs; ++i) {
    const int64_t s = lengths[i];
    if (s < 1 || s > kMaxLen) return HYDRA_ERR_INVALID;
    s_max = std::max(s_max, s);
    W += (u128)(s * s);
  }
  // ---- targets (Eq. (cstar-cont), (cstar), (load-target), (mstar))
  const int64_t c_mem = ceil2_d((double)s_max / (double)B);
  const double c_hat = cfg->pp > 1 ? (double)(s_max * s_max) *
                                          std::sqrt((double)(cfg->pp - 1) * cfg->theta_over_c * (double)G / (double)W)
                                    : 0.0;
  int64_t C;
  if (cfg->cap != 0) {
    C = cfg->cap;
  } else {
    const double want = std::max((double)c_mem, c_hat);
    C = want > (double)G ? G : std::min<int64_t>(G, ceil2_d(want));
  }
  if (C < 1 || (C & (C - 1)) != 0 || C > G || G % C != 0 || C < c_mem) return HYDRA_ERR_INVALID;
  const int64_t lam = s_max * s_max;  // Lambda* times C
  const int64_t budget = B * C;       // B times C
  const u128 num = (u128)C * W, den = (u128)(s_max * s_max) * (u128)G;
  const int64_t m_target = (int64_t)((num + den - 1) / den);
  const int levels = log2i(C);

  auto cp = [&](int64_t s) {
    int64_t k = 1;
    while (k < C && (k * lam < s * s * C || k * B < s)) k *= 2;
    return k;
  };

  std::vector<int64_t> order(n_docs);
  std::iota(order.begin(), order.end(), int64_t(0));
  std::stable_sort(order.begin(), order.end(), [&](int64_t a, int64_t b) { return lengths[a] > lengths[b]; });

  FreeRanks fr((int)G, levels);
  std::vector<Group> groups;
  std::vector<int32_t> doc_gid(n_docs, -1);
  std::vector<std::vector<int64_t>> members;
  std::vector<MinHeap<LoadEntry>> load_heap(levels + 1);
  std::vector<std::priority_queue<CapEntry>> cap_heap(levels + 1);
  std::vector<char> pruned(levels + 1, 0);
  int64_t max_load_all = 0;
  int32_t n_mbs = 0;
  int64_t pos = 0;

  while (pos < n_docs) {
    fr.reset();
    groups.clear();
    members.clear();
    for (int j = 0; j <= levels; ++j) {
      load_heap[j] = MinHeap<LoadEntry>();
      cap_heap[j] = std::priority_queue<CapEntry>();
      pruned[j] = 0;
    }
    MinHeap<MinLoad> min_heap;
    int64_t mb_max = 0;
    int64_t k_open = -1;
    while (pos < n_docs) {
      const int64_t d = order[pos], s = lengths[d];
      const int64_t k = cp(s);
      const int kl = log2i(k);
      int32_t gid = -1;
      const int32_t a = fr.lowest(kl);
      if (a >= 0) {  // a new k-aligned group on free ranks
        fr.take(a, (int32_t)k);
        gid = (int32_t)groups.size();
        groups.push_back(Group{a, (int32_t)k, 0, 0, 0});
        members.emplace_back();
        pruned[kl] = 0;
      } else {  // piggyback: smallest class first, least loaded (then lowest start) within it
        for (int j = kl; j <= levels && gid < 0; ++j) {
          if (pruned[j]) continue;
          const int64_t f = C >> j, dl = s * s * f, dt = s * f;
          auto& lh = load_heap[j];
          auto& ch = cap_heap[j];
          while (!ch.empty()) {  // re-admit groups whose capacity now covers the demand
            const CapEntry e = ch.top();
            const Group& g = groups[e.gid];
            if (e.ver != g.ver) { ch.pop(); continue; }
            if (e.remaining < dt) break;
            ch.pop();
            lh.push(LoadEntry{g.load, g.start, e.gid, g.ver});
          }
          while (!lh.empty()) {
            const LoadEntry e = lh.top();
            const Group& g = groups[e.gid];
            if (e.ver != g.ver) { lh.pop(); continue; }
            if (g.load >= lam) {  // the least loaded group is at the target
              if (ch.empty()) pruned[j] = 1;
              break;
            }
            if (g.load + dl > lam) break;
            if (g.tokens + dt > budget) {  // demote until its capacity covers the demand
              lh.pop();
              ch.push(CapEntry{budget - g.tokens, g.start, e.gid, g.ver});
              continue;
            }
            gid = e.gid;
            break;
          }
        }
      }
      if (gid < 0) break;  // nothing fits: close the micro-batch
      Group& g = groups[gid];
      const int64_t f = C / g.size;
      g.load += s * s * f;
      g.tokens += s * f;
      ++g.ver;
      load_heap[log2i(g.size)].push(LoadEntry{g.load, g.start, gid, g.ver});
      min_heap.push(MinLoad{g.load, gid, g.ver});
      mb_max = std::max(mb_max, g.load);
      doc_gid[d] = gid;
      members[gid].push_back(d);
      ++pos;
      if (k_open < 0) k_open = k;
      if (k < k_open && fr.free_count() == 0) {  // balance test (reading 3)
        while (min_heap.top().ver != groups[min_heap.top().gid].ver) min_heap.pop();
        if ((double)min_heap.top().load >= ratio * (double)mb_max) break;
      }
    }
    if (groups.empty()) return HYDRA_ERR_INVALID;  // unreachable: an empty MB takes any sequence
    // backfill idle ranks: double the smallest group whose buddy block is free
    MinHeap<SizeEntry> bf;
    for (int32_t i = 0; i < (int32_t)groups.size(); ++i) bf.push(SizeEntry{groups[i].size, groups[i].start, i});
    while (!bf.empty()) {
      const SizeEntry e = bf.top();
      bf.pop();
      Group& g = groups[e.gid];
      if (g.size != e.size || g.start != e.start) continue;
      if (2 * (int64_t)g.size > C) continue;
      const int32_t b = g.start ^ g.size;
      if (!fr.block_free(b, g.size)) continue;
      fr.take(b, g.size);
      g.start = std::min(g.start, b);
      g.size *= 2;
      g.load /= 2;
      g.tokens /= 2;
      bf.push(SizeEntry{g.size, g.start, e.gid});
    }
    for (int32_t i = 0; i < (int32_t)groups.size(); ++i) {
      max_load_all = std::max(max_load_all, groups[i].load);
      for (int64_t d : members[i]) {
        mb[d] = n_mbs;
        group_start[d] = groups[i].start;
        group_size[d] = groups[i].size;
      }
    }
    ++n_mbs;
  }
  if (summary) {
    summary->w_hi = (int64_t)(W >> 62);
    summary->w_lo = (int64_t)(W & ((u128(1) << 62) - 1));
    summary->s_max = s_max;
    summary->c_mem = (int32_t)c_mem;
    summary->c_hat = c_hat;
    summary->cap = (int32_t)C;
    summary->m_target = m_target;
    summary->n_mbs = n_mbs;
    summary->max_load_x_cap = max_load_all;
  }
  return HYDRA_OK;
}
