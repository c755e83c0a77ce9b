// The exported C ABI: validate on the host, plan, upload the plan, launch.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <initializer_list>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "hydra_attn.h"
#include "kernels.h"
#include "plan.h"
#include "prof.h"

namespace hydra {
hipError_t launch_attn_fwd(const AttnArgs& a, uint16_t* o_bf16, hipStream_t stream);
hipError_t launch_attn_bwd(const AttnArgs& a, int n_qitems, int n_kitems, const int* kitems, int kv_heads_per_pass,
                           hipStream_t stream);
hipError_t launch_lse_merge(int64_t n_rows, int H, float* o_acc, float* lse_acc, const float* o_part,
                            const float* lse_part, uint16_t* o_bf16, hipStream_t stream);
}  // namespace hydra

using namespace hydra;

// ------------------------------------------------------------------ kernel timing
namespace {
struct ProfRec {
  const char* name;
  hipEvent_t start, stop;
};
std::mutex g_prof_mu;
bool g_prof_on = false;
std::vector<ProfRec> g_prof;
}  // namespace

namespace hydra {
int prof_begin(const char* kernel, hipStream_t stream) {
  std::lock_guard<std::mutex> lock(g_prof_mu);
  if (!g_prof_on) return -1;
  ProfRec r{kernel, nullptr, nullptr};
  if (hipEventCreate(&r.start) != hipSuccess) return -1;
  if (hipEventCreate(&r.stop) != hipSuccess) {
    (void)hipEventDestroy(r.start);
    return -1;
  }
  (void)hipEventRecord(r.start, stream);
  g_prof.push_back(r);
  return int(g_prof.size()) - 1;
}
void prof_end(int token, hipStream_t stream) {
  if (token < 0) return;
  std::lock_guard<std::mutex> lock(g_prof_mu);
  if (token < int(g_prof.size())) (void)hipEventRecord(g_prof[token].stop, stream);
}
}  // namespace hydra

namespace {
void prof_clear_locked() {
  for (ProfRec& r : g_prof) {
    if (r.stop) (void)hipEventSynchronize(r.stop);
    (void)hipEventDestroy(r.start);
    (void)hipEventDestroy(r.stop);
  }
  g_prof.clear();
}
}  // namespace

namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// A device buffer as [p, p + n) bytes; NULL or empty spans overlap nothing.
struct Span {
  const void* p;
  uint64_t n;
};

bool overlap(Span a, Span b) {
  if (!a.p || !b.p || a.n == 0 || b.n == 0) return false;
  const uintptr_t x = reinterpret_cast<uintptr_t>(a.p), y = reinterpret_cast<uintptr_t>(b.p);
  return x < y + b.n && y < x + a.n;
}

// True if an output overlaps another output or any input (inputs may share memory).
bool outputs_overlap(std::initializer_list<Span> outs, std::initializer_list<Span> ins) {
  for (auto o = outs.begin(); o != outs.end(); ++o) {
    for (auto o2 = o + 1; o2 != outs.end(); ++o2)
      if (overlap(*o, *o2)) return true;
    for (const Span& i : ins)
      if (overlap(*o, i)) return true;
  }
  return false;
}

// Bytes from the first element of a bf16 token-major view to one past its last: `rows`
// rows of `width` elements, `stride` elements apart.
uint64_t rows_bytes(int64_t rows, int64_t stride, int64_t width) {
  return rows > 0 ? uint64_t((rows - 1) * stride + width) * 2 : 0;
}

// Non-null and 16-byte aligned when `needed`; HYDRA_OK otherwise.
int check_ptr(const void* p, bool needed) {
  if (!needed) return HYDRA_OK;
  if (!p) return HYDRA_ERR_INVALID;
  return aligned16(p) ? HYDRA_OK : HYDRA_ERR_ALIGN;
}

// Builds the host image of the workspace prefix (cu, query items, key items) and uploads it.
int upload_plan(const Problem& pr, const WsLayout& w, bool with_kv_items, void* ws, hipStream_t stream,
                std::vector<int32_t>* qitems, std::vector<int32_t>* kitems) {
  plan_items(pr, 0, qitems);
  if (with_kv_items) plan_items(pr, 1, kitems);
  const size_t bytes = with_kv_items ? w.d_off : w.kitems_off;
  std::vector<char> img(bytes, 0);
  std::memcpy(img.data() + w.cu_off, pr.cu.data(), pr.cu.size() * sizeof(int32_t));
  std::memcpy(img.data() + w.qitems_off, qitems->data(), qitems->size() * sizeof(int32_t));
  if (with_kv_items) {
    std::memcpy(img.data() + w.kitems_off, kitems->data(), kitems->size() * sizeof(int32_t));
    std::vector<int32_t> kbase, kmap32, krec;
    ds_tables(pr, *kitems, &kbase, &kmap32, &krec);
    std::memcpy(img.data() + w.kbase_off, kbase.data(), kbase.size() * sizeof(int32_t));
    std::memcpy(img.data() + w.kmap_off, kmap32.data(), kmap32.size() * sizeof(int32_t));
    std::memcpy(img.data() + w.krec_off, krec.data(), krec.size() * sizeof(int32_t));
  }
  // Pageable source: the runtime has consumed `img` when the call returns.
  if (hipMemcpyAsync(ws, img.data(), bytes, hipMemcpyHostToDevice, stream) != hipSuccess) return HYDRA_ERR_HIP;
  return HYDRA_OK;
}

// Which problem's plan each workspace holds, as far as this library uploaded it: the
// planned calls launch on the plan in the workspace, so they refuse a workspace whose
// plan was made for another problem (its row ranges would not fit the buffers) or that
// holds only the forward's query-side items.  Keyed by the workspace address; every
// upload through this library replaces the entry.
struct PlanRecord {
  std::vector<int64_t> key;  // what the plan depends on: heads, documents, both chunks
  bool has_kitems = false;
};
std::mutex g_plans_mu;
std::map<const void*, PlanRecord> g_plans;

std::vector<int64_t> plan_key(const Problem& pr) {
  std::vector<int64_t> k = {pr.H, pr.Hkv, int64_t(pr.cu.size())};
  k.insert(k.end(), pr.cu.begin(), pr.cu.end());
  for (const hydra_chunk_t* c : {&pr.q, &pr.kv}) {
    k.push_back(c->n_segs);
    for (int s = 0; s < c->n_segs; ++s) {
      k.push_back(c->start[s]);
      k.push_back(c->len[s]);
    }
  }
  return k;
}

void record_plan(const void* ws, const Problem& pr, bool has_kitems) {
  std::lock_guard<std::mutex> lock(g_plans_mu);
  PlanRecord& r = g_plans[ws];
  r.key = plan_key(pr);
  r.has_kitems = has_kitems;
}

// True if `ws` holds pr's plan, with the key-side items when `need_kitems`.
bool plan_matches(const void* ws, const Problem& pr, bool need_kitems) {
  std::lock_guard<std::mutex> lock(g_plans_mu);
  auto it = g_plans.find(ws);
  if (it == g_plans.end()) return false;
  if (need_kitems && !it->second.has_kitems) return false;
  return it->second.key == plan_key(pr);
}

AttnArgs base_args(const Problem& pr, const WsLayout& w, void* ws) {
  AttnArgs a{};
  char* base = static_cast<char*>(ws);
  a.cu = reinterpret_cast<const int*>(base + w.cu_off);
  a.items = reinterpret_cast<const int*>(base + w.qitems_off);
  a.Dvec = reinterpret_cast<float*>(base + w.d_off);
  a.lse2 = reinterpret_cast<float*>(base + w.lse2_off);
  a.kitems = reinterpret_cast<const int*>(base + w.kitems_off);
  a.kbase = reinterpret_cast<const int*>(base + w.kbase_off);
  a.kmap32 = reinterpret_cast<const int*>(base + w.kmap_off);
  a.krec = reinterpret_cast<const int*>(base + w.krec_off);
  a.n_docs = int(pr.cu.size()) - 1;
  a.H = pr.H;
  a.Hkv = pr.Hkv;
  a.grp = pr.H / pr.Hkv;
  a.kv_head0 = 0;
  a.kv_heads = pr.Hkv;
  a.q_head0 = 0;
  a.q_heads = pr.H;
  a.nq = int(pr.nq);
  a.nk = int(pr.nk);
  a.q_s = pr.q_s;
  a.k_s = pr.k_s;
  a.v_s = pr.v_s;
  a.scale = pr.scale;
  return a;
}

}  // namespace

extern "C" {

size_t hydra_workspace_size(const hydra_problem_t* p) {
  Problem pr;
  if (check_problem(p, &pr) != HYDRA_OK) return 0;
  return ws_layout(pr).total;
}

}  // extern "C"

namespace {

// Forward of one ring step; `upload` = false launches only (the plan is already in the
// workspace, from hydra_attn_plan).
int attn_fwd_impl(bool upload, const hydra_problem_t* p, const void* q, const void* k, const void* v, float* o_part,
                  float* lse_part, void* o_bf16, void* workspace, size_t workspace_bytes, void* stream) {
  try {
    Problem pr;
    int rc = check_problem(p, &pr);
    if (rc != HYDRA_OK) return rc;
    if (pr.nq == 0) return HYDRA_OK;
    const bool has_k = pr.nk > 0;
    for (int c : {check_ptr(q, true), check_ptr(k, has_k), check_ptr(v, has_k), check_ptr(o_part, true),
                  check_ptr(lse_part, true), o_bf16 ? check_ptr(o_bf16, true) : HYDRA_OK})
      if (c != HYDRA_OK) return c;
    const WsLayout w = ws_layout(pr);
    if (!workspace || workspace_bytes < w.total) return HYDRA_ERR_WORKSPACE;
    if (!aligned16(workspace)) return HYDRA_ERR_ALIGN;
    const uint64_t qh = uint64_t(pr.nq) * pr.H;
    const uint64_t qb = rows_bytes(pr.nq, pr.q_s, pr.H * kDqk), kb = rows_bytes(pr.nk, pr.k_s, pr.Hkv * kDqk),
                   vb = rows_bytes(pr.nk, pr.v_s, pr.Hkv * kDv);
    if (outputs_overlap({{o_part, qh * kDv * 4}, {lse_part, qh * 4}, {o_bf16, qh * kDv * 2}, {workspace, w.total}},
                        {{q, qb}, {k, kb}, {v, vb}}))
      return HYDRA_ERR_INVALID;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (upload) {  // the forward needs only the query-stationary items
      std::vector<int32_t> qitems, kitems;
      rc = upload_plan(pr, w, false, workspace, s, &qitems, &kitems);
      if (rc != HYDRA_OK) return rc;
      record_plan(workspace, pr, false);
    } else if (!plan_matches(workspace, pr, false)) {
      return HYDRA_ERR_WORKSPACE;
    }
    AttnArgs a = base_args(pr, w, workspace);
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k);
    a.v = static_cast<const uint16_t*>(v);
    a.out_o = o_part;
    a.out_lse = lse_part;
    a.n_items = int(w.n_qitems);
    if (launch_attn_fwd(a, static_cast<uint16_t*>(o_bf16), s) != hipSuccess) return HYDRA_ERR_HIP;
    return HYDRA_OK;
  } catch (...) {
    return HYDRA_ERR_INVALID;
  }
}

// Bytes of stored dS per query head on the stored-dS path (0 when the path does not apply).
uint64_t ds_bytes_per_head(const Problem& pr) {
  if (!ds_path_applies(pr)) return 0;
  std::vector<int32_t> kitems, kbase, kmap32, krec;
  plan_items(pr, 1, &kitems);
  return uint64_t(ds_tables(pr, kitems, &kbase, &kmap32, &krec)) * DS_TILE_BYTES;
}

int attn_bwd_impl(bool upload, const hydra_problem_t* p, const void* q, const void* k, const void* v,
                  const void* o_final, const float* lse_final, const void* d_o, float* dq_acc, float* dk_acc,
                  float* dv_acc, void* ds_buf, size_t ds_bytes, void* workspace, size_t workspace_bytes,
                  void* stream) {
  try {
    Problem pr;
    int rc = check_problem(p, &pr);
    if (rc != HYDRA_OK) return rc;
    if (pr.nq == 0 || pr.nk == 0) return HYDRA_OK;
    for (int c : {check_ptr(q, true), check_ptr(k, true), check_ptr(v, true), check_ptr(o_final, true),
                  check_ptr(lse_final, true), check_ptr(d_o, true), check_ptr(dq_acc, true),
                  check_ptr(dk_acc, true), check_ptr(dv_acc, true)})
      if (c != HYDRA_OK) return c;
    const WsLayout w = ws_layout(pr);
    if (!workspace || workspace_bytes < w.total) return HYDRA_ERR_WORKSPACE;
    if (!aligned16(workspace)) return HYDRA_ERR_ALIGN;
    // stored-dS path: K/V heads per pass such that their query heads' dS fits ds_buf
    int kv_per_pass = 0;
    uint64_t ds_head = 0;
    if (ds_buf) {
      if (!aligned16(ds_buf)) return HYDRA_ERR_ALIGN;
      ds_head = ds_bytes_per_head(pr);
      const uint64_t per_kv = ds_head * uint64_t(pr.H / pr.Hkv);
      if (per_kv > 0) kv_per_pass = int(std::min<uint64_t>(uint64_t(pr.Hkv), uint64_t(ds_bytes) / per_kv));
    }
    const uint64_t ds_used = uint64_t(kv_per_pass) * (pr.H / pr.Hkv) * ds_head;
    const uint64_t qh = uint64_t(pr.nq) * pr.H, kh = uint64_t(pr.nk) * pr.Hkv;
    const uint64_t qb = rows_bytes(pr.nq, pr.q_s, pr.H * kDqk), kb = rows_bytes(pr.nk, pr.k_s, pr.Hkv * kDqk),
                   vb = rows_bytes(pr.nk, pr.v_s, pr.Hkv * kDv);
    if (outputs_overlap({{dq_acc, qh * kDqk * 4}, {dk_acc, kh * kDqk * 4}, {dv_acc, kh * kDv * 4},
                         {workspace, w.total}, {kv_per_pass ? ds_buf : nullptr, ds_used}},
                        {{q, qb}, {k, kb}, {v, vb}, {o_final, qh * kDv * 2}, {lse_final, qh * 4},
                         {d_o, qh * kDv * 2}}))
      return HYDRA_ERR_INVALID;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (upload) {
      std::vector<int32_t> qitems, kitems;
      rc = upload_plan(pr, w, true, workspace, s, &qitems, &kitems);
      if (rc != HYDRA_OK) return rc;
      record_plan(workspace, pr, true);
    } else if (!plan_matches(workspace, pr, true)) {
      return HYDRA_ERR_WORKSPACE;
    }
    AttnArgs a = base_args(pr, w, workspace);
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k);
    a.v = static_cast<const uint16_t*>(v);
    a.o = static_cast<const uint16_t*>(o_final);
    a.dO = static_cast<const uint16_t*>(d_o);
    a.lse = lse_final;
    a.dq = dq_acc;
    a.dk = dk_acc;
    a.dv = dv_acc;
    a.ds = static_cast<char*>(kv_per_pass ? ds_buf : nullptr);
    a.ds_head_bytes = int64_t(ds_head);
    const int* kitems_dev = reinterpret_cast<const int*>(static_cast<char*>(workspace) + w.kitems_off);
    if (launch_attn_bwd(a, int(w.n_qitems), int(w.n_kitems), kitems_dev, kv_per_pass, s) != hipSuccess)
      return HYDRA_ERR_HIP;
    return HYDRA_OK;
  } catch (...) {
    return HYDRA_ERR_INVALID;
  }
}

}  // namespace

extern "C" {

int hydra_attn_plan(const hydra_problem_t* p, void* workspace, size_t workspace_bytes, void* stream) {
  try {
    Problem pr;
    int rc = check_problem(p, &pr);
    if (rc != HYDRA_OK) return rc;
    const WsLayout w = ws_layout(pr);
    if (!workspace || workspace_bytes < w.total) return HYDRA_ERR_WORKSPACE;
    if (!aligned16(workspace)) return HYDRA_ERR_ALIGN;
    std::vector<int32_t> qitems, kitems;
    rc = upload_plan(pr, w, true, workspace, static_cast<hipStream_t>(stream), &qitems, &kitems);
    if (rc == HYDRA_OK) record_plan(workspace, pr, true);
    return rc;
  } catch (...) {
    return HYDRA_ERR_INVALID;
  }
}

int hydra_attn_fwd(const hydra_problem_t* p, const void* q, const void* k, const void* v, float* o_part,
                   float* lse_part, void* o_bf16, void* workspace, size_t workspace_bytes, void* stream) {
  return attn_fwd_impl(true, p, q, k, v, o_part, lse_part, o_bf16, workspace, workspace_bytes, stream);
}

int hydra_attn_fwd_planned(const hydra_problem_t* p, const void* q, const void* k, const void* v, float* o_part,
                           float* lse_part, void* o_bf16, void* workspace, size_t workspace_bytes, void* stream) {
  return attn_fwd_impl(false, p, q, k, v, o_part, lse_part, o_bf16, workspace, workspace_bytes, stream);
}

int hydra_attn_bwd(const hydra_problem_t* p, const void* q, const void* k, const void* v, const void* o_final,
                   const float* lse_final, const void* d_o, float* dq_acc, float* dk_acc, float* dv_acc,
                   void* workspace, size_t workspace_bytes, void* stream) {
  return attn_bwd_impl(true, p, q, k, v, o_final, lse_final, d_o, dq_acc, dk_acc, dv_acc, nullptr, 0, workspace,
                       workspace_bytes, stream);
}

int hydra_attn_bwd_ds(const hydra_problem_t* p, const void* q, const void* k, const void* v, const void* o_final,
                      const float* lse_final, const void* d_o, float* dq_acc, float* dk_acc, float* dv_acc,
                      void* ds_buf, size_t ds_bytes, void* workspace, size_t workspace_bytes, void* stream) {
  return attn_bwd_impl(true, p, q, k, v, o_final, lse_final, d_o, dq_acc, dk_acc, dv_acc, ds_buf, ds_bytes,
                       workspace, workspace_bytes, stream);
}

}  // extern "C"

// ------------------------------------------------------------------ the no-allocation backward
// For callers that cannot allocate device memory (code under stream capture, tight serving
// loops): the backward's workspace (plan, D, LSE*log2(e)) lives in this file-scope array
// instead, one copy per GPU, held until the process ends.  Host code never passes the
// array's name to a kernel or a copy (on the host it is only a stand-in for the symbol):
// each device's address comes from hipGetSymbolAddress, once per device, with that device
// current.
namespace {
constexpr size_t kNoAllocScratchBytes = size_t(32) << 20;  // 32 MiB
static __device__ __align__(256) char scratch[kNoAllocScratchBytes];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's copy of `scratch`, looked up on its first use.
int scratch_ptr(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return HYDRA_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return HYDRA_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return HYDRA_OK;
}
}  // namespace

extern "C" {

size_t hydra_noalloc_scratch_bytes(void) { return kNoAllocScratchBytes; }

int hydra_attn_bwd_noalloc(const hydra_problem_t* p, const void* q, const void* k, const void* v,
                           const void* o_final, const float* lse_final, const void* d_o, float* dq_acc,
                           float* dk_acc, float* dv_acc, void* stream) {
  try {
    Problem pr;
    int rc = check_problem(p, &pr);
    if (rc != HYDRA_OK) return rc;
    if (ws_layout(pr).total > kNoAllocScratchBytes) return HYDRA_ERR_TOO_LARGE;
    void* ws = nullptr;
    if ((rc = scratch_ptr(&ws)) != HYDRA_OK) return rc;
    return attn_bwd_impl(true, p, q, k, v, o_final, lse_final, d_o, dq_acc, dk_acc, dv_acc, nullptr, 0, ws,
                         kNoAllocScratchBytes, stream);
  } catch (...) {
    return HYDRA_ERR_INVALID;
  }
}

size_t hydra_bwd_ds_bytes(const hydra_problem_t* p, int32_t kv_heads_per_pass) {
  try {
    Problem pr;
    if (check_problem(p, &pr) != HYDRA_OK || kv_heads_per_pass < 1) return 0;
    const uint64_t per_head = ds_bytes_per_head(pr);
    return size_t(per_head * uint64_t(std::min(kv_heads_per_pass, pr.Hkv)) * uint64_t(pr.H / pr.Hkv));
  } catch (...) {
    return 0;
  }
}

int hydra_attn_bwd_planned(const hydra_problem_t* p, const void* q, const void* k, const void* v,
                           const void* o_final, const float* lse_final, const void* d_o, float* dq_acc,
                           float* dk_acc, float* dv_acc, void* workspace, size_t workspace_bytes, void* stream) {
  return attn_bwd_impl(false, p, q, k, v, o_final, lse_final, d_o, dq_acc, dk_acc, dv_acc, nullptr, 0, workspace,
                       workspace_bytes, stream);
}

int hydra_lse_merge(int64_t n_rows, int32_t n_heads, int32_t d_v, float* o_acc, float* lse_acc,
                    const float* o_part, const float* lse_part, void* o_out_bf16, void* stream) {
  if (n_rows < 0 || n_heads <= 0 || n_heads > 4096) return HYDRA_ERR_INVALID;
  if (d_v != kDv) return d_v <= 0 ? HYDRA_ERR_INVALID : HYDRA_ERR_UNSUPPORTED;
  if (n_rows > (int64_t(1) << 30)) return HYDRA_ERR_INVALID;
  if (n_rows == 0) return HYDRA_OK;
  for (int c : {check_ptr(o_acc, true), check_ptr(lse_acc, true), check_ptr(o_part, true),
                check_ptr(lse_part, true), o_out_bf16 ? check_ptr(o_out_bf16, true) : HYDRA_OK})
    if (c != HYDRA_OK) return c;
  const uint64_t rh = uint64_t(n_rows) * uint64_t(n_heads);
  if (outputs_overlap({{o_acc, rh * kDv * 4}, {lse_acc, rh * 4}, {o_out_bf16, rh * kDv * 2}},
                      {{o_part, rh * kDv * 4}, {lse_part, rh * 4}}))
    return HYDRA_ERR_INVALID;
  if (launch_lse_merge(n_rows, n_heads, o_acc, lse_acc, o_part, lse_part, static_cast<uint16_t*>(o_out_bf16),
                       static_cast<hipStream_t>(stream)) != hipSuccess)
    return HYDRA_ERR_HIP;
  return HYDRA_OK;
}

const char* hydra_strerror(int status) {
  switch (status) {
    case HYDRA_OK: return "ok";
    case HYDRA_ERR_INVALID: return "invalid argument";
    case HYDRA_ERR_UNSUPPORTED: return "unsupported problem (d_qk must be 192 and d_v 128)";
    case HYDRA_ERR_ALIGN: return "device pointer not 16-byte aligned";
    case HYDRA_ERR_WORKSPACE: return "workspace missing or too small";
    case HYDRA_ERR_HIP: return "HIP runtime error";
    case HYDRA_ERR_TOO_LARGE:
      return "problem needs more workspace than the no-allocation call's 32 MiB scratch holds";
    default: return "unknown status";
  }
}

int64_t hydra_visible_pairs(const hydra_problem_t* p) {
  Problem pr;
  if (check_problem(p, &pr) != HYDRA_OK) return -1;
  return visible_pairs(pr);
}

int64_t hydra_plan_items(const hydra_problem_t* p, int32_t which, int32_t* out, int64_t cap) {
  Problem pr;
  int rc = check_problem(p, &pr);
  if (rc != HYDRA_OK) return rc;
  if (which != 0 && which != 1) return HYDRA_ERR_INVALID;
  if (cap < 0 || (cap > 0 && !out)) return HYDRA_ERR_INVALID;
  std::vector<int32_t> items;
  plan_items(pr, which, &items);
  const int64_t n = int64_t(items.size()) / kItemInts;
  const int64_t k = n < cap ? n : cap;
  if (k > 0) std::memcpy(out, items.data(), size_t(k) * kItemInts * sizeof(int32_t));
  return n;
}

int hydra_profile_start(void) {
  std::lock_guard<std::mutex> lock(g_prof_mu);
  prof_clear_locked();
  g_prof_on = true;
  return HYDRA_OK;
}

int hydra_profile_stop(hydra_kernel_stat_t* out, int32_t cap) {
  std::lock_guard<std::mutex> lock(g_prof_mu);
  g_prof_on = false;
  if (cap < 0 || (cap > 0 && !out)) return HYDRA_ERR_INVALID;
  std::map<std::string, hydra_kernel_stat_t> agg;
  int status = HYDRA_OK;
  for (ProfRec& r : g_prof) {
    float ms = 0.f;
    if (hipEventSynchronize(r.stop) != hipSuccess || hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess) {
      status = HYDRA_ERR_HIP;
      continue;
    }
    hydra_kernel_stat_t& k = agg[r.name];
    if (k.launches == 0) {
      std::memset(&k, 0, sizeof(k));
      std::strncpy(k.name, r.name, sizeof(k.name) - 1);
      k.min_ms = ms;
      k.max_ms = ms;
    }
    k.launches += 1;
    k.total_ms += ms;
    k.min_ms = std::min<double>(k.min_ms, ms);
    k.max_ms = std::max<double>(k.max_ms, ms);
  }
  prof_clear_locked();
  if (status != HYDRA_OK) return status;
  int n = 0;
  for (auto& kv : agg) {
    if (n < cap) out[n] = kv.second;
    ++n;
  }
  return n;
}

void hydra_tile_rows(int32_t* q_tile_rows, int32_t* kv_tile_rows) {
  if (q_tile_rows) *q_tile_rows = kQTile;
  if (kv_tile_rows) *kv_tile_rows = kKvTile;
}

}  // extern "C"
