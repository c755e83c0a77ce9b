// Host-side argument checks and work planning for one ring step.
//
// The plan cuts each side of a ring step into tiles that never straddle a segment, so
// the rows of a tile are consecutive global positions.  For a query tile with positions
// [a, b] the visible keys form one contiguous position interval, [doc_start(a), b]: the
// union over its rows p of [doc_start(p), p] has no gaps because document starts only
// grow with p.  Symmetrically, a key tile [a, b] is seen by the query interval
// [a, doc_end(b) - 1].  Intersecting that interval with each segment of the other chunk
// gives at most HYDRA_MAX_SEGS contiguous ranges of local rows; anything outside them is
// masked (Sec. 2.2) and is never visited.  Tiles are ordered heaviest first, the
// kernel-level counterpart of the scheduler placing the longest sequences first
// (Sec. 5.1.1, Alg. 1, phase 2).
#include "plan.h"

#include "tiles.h"

#include <algorithm>
#include <cmath>
#include <numeric>

namespace hydra {

namespace {

constexpr int64_t kMaxRows = int64_t(1) << 30;

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

int64_t chunk_rows(const hydra_chunk_t& c) {
  int64_t n = 0;
  for (int s = 0; s < c.n_segs; ++s) n += c.len[s];
  return n;
}

int check_chunk(const hydra_chunk_t& c, int64_t total) {
  if (c.n_segs < 0 || c.n_segs > HYDRA_MAX_SEGS) return HYDRA_ERR_INVALID;
  for (int s = 0; s < c.n_segs; ++s) {
    if (c.start[s] < 0 || c.len[s] < 0) return HYDRA_ERR_INVALID;
    if (int64_t(c.start[s]) + c.len[s] > total) return HYDRA_ERR_INVALID;
  }
  return HYDRA_OK;
}

// Index d with cu[d] <= pos < cu[d+1] (pos inside the packed window).
int doc_index(const std::vector<int32_t>& cu, int64_t pos) {
  auto it = std::upper_bound(cu.begin(), cu.end(), int32_t(pos));
  return int(it - cu.begin()) - 1;
}

struct Tile {
  int32_t row0, pos0, n;
};

void tiles_of(const hydra_chunk_t& c, int rows_per_tile, std::vector<Tile>* out) {
  int32_t row = 0;
  for (int s = 0; s < c.n_segs; ++s) {
    for (int32_t t = 0; t < c.len[s]; t += rows_per_tile)
      out->push_back({row + t, c.start[s] + t, std::min<int32_t>(rows_per_tile, c.len[s] - t)});
    row += c.len[s];
  }
}

// Ranges of local rows of chunk `c` whose positions fall in [lo, hi] (inclusive).
int ranges_in(const hydra_chunk_t& c, int64_t lo, int64_t hi, int32_t* dst) {
  int n = 0;
  int32_t row = 0;
  for (int s = 0; s < c.n_segs; ++s) {
    int64_t a = std::max<int64_t>(lo, c.start[s]);
    int64_t b = std::min<int64_t>(hi, int64_t(c.start[s]) + c.len[s] - 1);
    if (a <= b) {
      dst[3 * n + 0] = row + int32_t(a - c.start[s]);
      dst[3 * n + 1] = int32_t(a);
      dst[3 * n + 2] = int32_t(b - a + 1);
      ++n;
    }
    row += c.len[s];
  }
  return n;
}

// Pairs (p, k) with p in [qa, qb), k in [ka, kb), k <= p.
int64_t causal_pairs(int64_t qa, int64_t qb, int64_t ka, int64_t kb) {
  if (qb <= qa || kb <= ka) return 0;
  int64_t total = 0;
  int64_t a = std::max(qa, ka), b = std::min(qb, kb);
  if (b > a) {
    int64_t hi = b - ka, lo = a - ka;  // sum of x for x in (lo, hi]
    total += hi * (hi + 1) / 2 - lo * (lo + 1) / 2;
  }
  int64_t full = qb - std::max(qa, kb);
  if (full > 0) total += full * (kb - ka);
  return total;
}

}  // namespace

int check_problem(const hydra_problem_t* p, Problem* out) {
  if (!p || !out) return HYDRA_ERR_INVALID;
  if (p->n_heads <= 0 || p->n_heads > 4096) return HYDRA_ERR_INVALID;
  if (p->d_qk <= 0 || p->d_v <= 0) return HYDRA_ERR_INVALID;
  if (p->d_qk != kDqk || p->d_v != kDv) return HYDRA_ERR_UNSUPPORTED;
  if (!std::isfinite(p->softmax_scale)) return HYDRA_ERR_INVALID;
  if (!p->cu_seqlens || p->n_docs < 1) return HYDRA_ERR_INVALID;
  if (p->cu_seqlens[0] != 0) return HYDRA_ERR_INVALID;
  for (int d = 0; d < p->n_docs; ++d)
    if (p->cu_seqlens[d + 1] < p->cu_seqlens[d]) return HYDRA_ERR_INVALID;
  const int64_t total = p->cu_seqlens[p->n_docs];
  int rc = check_chunk(p->q, total);
  if (rc != HYDRA_OK) return rc;
  rc = check_chunk(p->kv, total);
  if (rc != HYDRA_OK) return rc;
  const int64_t nq = chunk_rows(p->q), nk = chunk_rows(p->kv);
  if (nq > kMaxRows || nk > kMaxRows) return HYDRA_ERR_INVALID;
  if (nq * p->n_heads * kDqk >= (int64_t(1) << 40) || nk * p->n_heads * kDqk >= (int64_t(1) << 40))
    return HYDRA_ERR_INVALID;
  const int hkv = p->n_kv_heads == 0 ? p->n_heads : p->n_kv_heads;
  if (hkv < 0 || hkv > p->n_heads || p->n_heads % hkv != 0) return HYDRA_ERR_INVALID;
  if (nk * hkv * kDqk >= (int64_t(1) << 40)) return HYDRA_ERR_INVALID;
  // The attention launches have one 512-lane workgroup per (tile, head), and a dispatch
  // holds fewer than 2^32 lanes.
  int64_t nqt = 0, nkt = 0;
  for (int s = 0; s < p->q.n_segs; ++s) nqt += (p->q.len[s] + kQTile - 1) / kQTile;
  for (int s = 0; s < p->kv.n_segs; ++s) nkt += (p->kv.len[s] + kKvTile - 1) / kKvTile;
  if (nqt * p->n_heads >= (int64_t(1) << 23) || nkt * hkv >= (int64_t(1) << 23)) return HYDRA_ERR_INVALID;
  // token-row strides: 0 = dense; else >= dense, a multiple of 8 (16-byte rows), < 2^22
  auto stride = [](int32_t s, int64_t dense, int* dst) {
    if (s == 0) s = int32_t(dense);
    if (s < dense || s % 8 != 0 || s >= (1 << 22)) return false;
    *dst = s;
    return true;
  };
  if (!stride(p->q_tok_stride, int64_t(p->n_heads) * kDqk, &out->q_s) ||
      !stride(p->k_tok_stride, int64_t(hkv) * kDqk, &out->k_s) ||
      !stride(p->v_tok_stride, int64_t(hkv) * kDv, &out->v_s))
    return HYDRA_ERR_INVALID;
  if (nq * out->q_s >= (int64_t(1) << 40) || nk * out->k_s >= (int64_t(1) << 40)) return HYDRA_ERR_INVALID;
  out->H = p->n_heads;
  out->Hkv = hkv;
  out->scale = p->softmax_scale > 0.f ? p->softmax_scale : 1.0f / std::sqrt(float(kDqk));
  out->cu.assign(p->cu_seqlens, p->cu_seqlens + p->n_docs + 1);
  out->q = p->q;
  out->kv = p->kv;
  out->nq = nq;
  out->nk = nk;
  return HYDRA_OK;
}

void plan_items(const Problem& pr, int which, std::vector<int32_t>* items) {
  const hydra_chunk_t& own = which == 0 ? pr.q : pr.kv;
  const hydra_chunk_t& other = which == 0 ? pr.kv : pr.q;
  std::vector<Tile> tiles;
  tiles_of(own, which == 0 ? kQTile : kKvTile, &tiles);
  const size_t n = tiles.size();
  std::vector<int32_t> raw(n * kItemInts, 0);
  std::vector<int64_t> cost(n, 0);
  for (size_t i = 0; i < n; ++i) {
    const Tile& t = tiles[i];
    int32_t* it = &raw[i * kItemInts];
    it[0] = t.row0;
    it[1] = t.pos0;
    it[2] = t.n;
    const int64_t first = t.pos0, last = int64_t(t.pos0) + t.n - 1;
    int64_t lo, hi;
    if (which == 0) {  // keys seen by queries [first, last]
      lo = pr.cu[doc_index(pr.cu, first)];
      hi = last;
    } else {           // queries that see keys [first, last]
      lo = first;
      hi = int64_t(pr.cu[doc_index(pr.cu, last) + 1]) - 1;
    }
    it[3] = ranges_in(other, lo, hi, it + 4);
    for (int r = 0; r < it[3]; ++r) cost[i] += it[4 + 3 * r + 2];
  }
  std::vector<size_t> order(n);
  std::iota(order.begin(), order.end(), size_t(0));
  std::stable_sort(order.begin(), order.end(), [&](size_t a, size_t b) { return cost[a] > cost[b]; });
  items->resize(n * kItemInts);
  for (size_t i = 0; i < n; ++i)
    std::copy(&raw[order[i] * kItemInts], &raw[order[i] * kItemInts] + kItemInts, &(*items)[i * kItemInts]);
}

int64_t visible_pairs(const Problem& pr) {
  int64_t total = 0;
  const int n_docs = int(pr.cu.size()) - 1;
  for (int qs = 0; qs < pr.q.n_segs; ++qs) {
    const int64_t qa = pr.q.start[qs], qb = qa + pr.q.len[qs];
    if (qb <= qa) continue;
    for (int ks = 0; ks < pr.kv.n_segs; ++ks) {
      const int64_t ka = pr.kv.start[ks], kb = ka + pr.kv.len[ks];
      if (kb <= ka) continue;
      // documents overlapping the query segment
      int d0 = doc_index(pr.cu, qa), d1 = doc_index(pr.cu, qb - 1);
      for (int d = std::max(d0, 0); d <= d1 && d < n_docs; ++d) {
        const int64_t da = pr.cu[d], db = pr.cu[d + 1];
        total += causal_pairs(std::max(qa, da), std::min(qb, db), std::max(ka, da), std::min(kb, db));
      }
    }
  }
  return total;
}

bool ds_path_applies(const Problem& pr) {
  if (pr.nq == 0 || pr.nk == 0) return false;
  for (const hydra_chunk_t* c : {&pr.q, &pr.kv})
    for (int s = 0; s < c->n_segs; ++s)
      if (c->start[s] % 32 != 0 || c->len[s] % 32 != 0) return false;
  return true;
}

int64_t ds_tables(const Problem& pr, const std::vector<int32_t>& kitems, std::vector<int32_t>* kbase,
                  std::vector<int32_t>* kmap32, std::vector<int32_t>* krec) {
  const int64_t n = int64_t(kitems.size()) / kItemInts;
  kbase->assign(size_t(n), 0);
  kmap32->assign(size_t((pr.nk + 31) / 32), -1);
  krec->assign(size_t(n) * kItemInts, 0);
  std::vector<int64_t> order(static_cast<size_t>(n));
  std::iota(order.begin(), order.end(), int64_t(0));
  std::sort(order.begin(), order.end(),
            [&](int64_t x, int64_t y) { return kitems[size_t(x) * kItemInts] < kitems[size_t(y) * kItemInts]; });
  int64_t slots = 0;
  for (int64_t i = 0; i < n; ++i) {
    const int32_t* it = &kitems[size_t(i) * kItemInts];
    (*kbase)[size_t(i)] = int32_t(slots);
    for (int r = 0; r < it[3]; ++r) slots += (it[4 + 3 * r + 2] + KV_QTILE_ROWS - 1) / KV_QTILE_ROWS;
  }
  for (int64_t j = 0; j < n; ++j) {
    const int64_t i = order[size_t(j)];
    const int32_t* it = &kitems[size_t(i) * kItemInts];
    int32_t* rec = &(*krec)[size_t(j) * kItemInts];
    rec[0] = it[0];
    rec[1] = it[2];
    rec[2] = it[3];
    rec[3] = (*kbase)[size_t(i)];
    for (int r = 0; r < it[3]; ++r) {
      rec[4 + 2 * r] = it[4 + 3 * r];
      rec[5 + 2 * r] = it[6 + 3 * r];
    }
    for (int32_t b = it[0] / 32; b < (it[0] + it[2] + 31) / 32; ++b) (*kmap32)[size_t(b)] = int32_t(j);
  }
  return slots;
}

WsLayout ws_layout(const Problem& pr) {
  WsLayout w{};
  const int64_t nqt = [&] {
    int64_t n = 0;
    for (int s = 0; s < pr.q.n_segs; ++s) n += (pr.q.len[s] + kQTile - 1) / kQTile;
    return n;
  }();
  const int64_t nkt = [&] {
    int64_t n = 0;
    for (int s = 0; s < pr.kv.n_segs; ++s) n += (pr.kv.len[s] + kKvTile - 1) / kKvTile;
    return n;
  }();
  w.n_qitems = nqt;
  w.n_kitems = nkt;
  size_t off = 0;
  w.cu_off = off;
  off = align_up(off + pr.cu.size() * sizeof(int32_t), 256);
  w.qitems_off = off;
  off = align_up(off + size_t(nqt) * kItemInts * sizeof(int32_t), 256);
  w.kitems_off = off;
  off = align_up(off + size_t(nkt) * kItemInts * sizeof(int32_t), 256);
  w.n_kblocks = (pr.nk + 31) / 32;
  w.kbase_off = off;
  off = align_up(off + size_t(nkt) * sizeof(int32_t), 256);
  w.kmap_off = off;
  off = align_up(off + size_t(w.n_kblocks) * sizeof(int32_t), 256);
  w.krec_off = off;
  off = align_up(off + size_t(nkt) * kItemInts * sizeof(int32_t), 256);
  w.d_off = off;
  off = align_up(off + size_t(pr.H) * size_t(pr.nq) * sizeof(float), 256);
  w.lse2_off = off;
  off = align_up(off + size_t(pr.H) * size_t(pr.nq) * sizeof(float), 256);
  w.total = std::max<size_t>(off, 256);
  return w;
}

}  // namespace hydra
