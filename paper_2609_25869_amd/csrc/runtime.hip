// C-ABI of the block-sparse attention library: request validation, the
// online request path of Algorithm 2 (mu(M) on the GPU, one statistics copy
// to the host, regime lookup, ranked fallback, launch preparation of the
// selected plan only) and plan execution (Section 3).
#include <dlfcn.h>

#include <climits>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <fstream>
#include <map>
#include <memory>
#include <mutex>
#include <sstream>
#include <algorithm>
#include <string>
#include <vector>

#include "../../include/bsa.h"
#include "bsa_internal.h"
#include "catalog.h"
#include "slot_map.h"

using namespace bsa;

namespace {

thread_local std::string g_err;

bsa_status fail(bsa_status s, const std::string& msg) {
  g_err = msg;
  if (std::getenv("BSA_LOG")) std::fprintf(stderr, "[bsa] error: %s\n", msg.c_str());
  return s;
}

#define HIP_TRY(expr)                                                                              \
  do {                                                                                             \
    hipError_t e_ = (expr);                                                                        \
    if (e_ != hipSuccess) return fail(BSA_ERR_HIP, std::string(#expr) + ": " + hipGetErrorString(e_)); \
  } while (0)

bool log_on() { return std::getenv("BSA_LOG") != nullptr; }

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

int ilog2_exact(int64_t x) {
  int s = 0;
  while ((int64_t(1) << s) < x) ++s;
  return ((int64_t(1) << s) == x) ? s : -1;
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Task count above which the planner sorts a segment's tasks into KV order.
constexpr int64_t kOrderMinTasks = 512;

// Length of the runs of consecutive tasks that the XCDs of one group take
// turns over (see the plan's traversal order, CatalogEntry::xcd_group).
constexpr int32_t kSlotRun = 8;

// ---------------------------------------------------------------------------
// Pinned staging for the per-request host<->device copies.  One buffer per
// process, reused; the lock is held from the upload until the request's one
// synchronisation, after which the copies are complete.
struct Staging {
  std::mutex mu;
  void* ptr = nullptr;
  size_t bytes = 0;
  bsa_status reserve(size_t need) {
    if (need <= bytes) return BSA_OK;
    if (ptr) (void)hipHostFree(ptr);
    ptr = nullptr;
    bytes = 0;
    size_t cap = need < (1 << 20) ? (1 << 20) : need * 2;
    if (hipHostMalloc(&ptr, cap, hipHostMallocDefault) != hipSuccess) {
      ptr = nullptr;
      return fail(BSA_ERR_OOM, "pinned host staging allocation failed");
    }
    bytes = cap;
    return BSA_OK;
  }
};
Staging& staging() {
  static Staging* s = new Staging();  // intentionally leaked: lives to process exit
  return *s;
}

// Stream-ordered device memory: keep freed blocks in the pool so repeated
// requests do not return memory to the driver.
std::mutex g_pool_mu;
std::map<int, bool> g_pool_ready;
void prepare_pool(int dev) {
  std::lock_guard<std::mutex> lk(g_pool_mu);
  if (g_pool_ready[dev]) return;
  hipMemPool_t pool;
  if (hipDeviceGetDefaultMemPool(&pool, dev) == hipSuccess) {
    uint64_t thr = UINT64_MAX;
    (void)hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &thr);
  }
  g_pool_ready[dev] = true;
}

// ---------------------------------------------------------------------------
// Default plan table: BSA_LUT_PATH, else lut/gfx950_v1.json beside the library.
std::once_flag g_lut_once;
Lut* g_default_lut = nullptr;
std::string g_default_lut_msg;

std::string library_dir() {
  Dl_info info;
  if (dladdr(reinterpret_cast<void*>(&bsa_version), &info) && info.dli_fname) {
    std::string p = info.dli_fname;
    size_t k = p.find_last_of('/');
    return k == std::string::npos ? std::string(".") : p.substr(0, k);
  }
  return ".";
}

bool read_file(const std::string& path, std::string* out) {
  std::ifstream f(path, std::ios::binary);
  if (!f) return false;
  std::ostringstream ss;
  ss << f.rdbuf();
  *out = ss.str();
  return true;
}

const Lut* default_lut() {
  std::call_once(g_lut_once, [] {
    const char* env = std::getenv("BSA_LUT_PATH");
    std::string path = env ? env : library_dir() + "/lut/gfx950_v1.json";
    std::string text, err;
    if (!read_file(path, &text)) {
      g_default_lut_msg = "no plan table at " + path + "; base plans only";
    } else {
      Lut* l = new Lut();
      if (lut_parse(text, l, &err)) {
        g_default_lut = l;
        g_default_lut_msg = "plan table " + path;
      } else {
        delete l;
        g_default_lut_msg = "plan table " + path + " rejected (" + err + "); base plans only";
      }
    }
    if (log_on()) std::fprintf(stderr, "[bsa] %s\n", g_default_lut_msg.c_str());
  });
  return g_default_lut;
}

}  // namespace

struct bsa_lut_s {
  Lut lut;
};

// ---------------------------------------------------------------------------
// Plan object

namespace {

struct Segment {
  int32_t bq = 0, bkv = 0;
  std::vector<int32_t> heads;
  int32_t seg_heads_off = 0;  // offset of this segment's head list in the device table
  CatalogEntry plan{};
  int32_t mapping = 0;
  bool regime_hit = false;
  int64_t nnz = 0, blocks = 0, run_blocks = 0, max_row_nnz = 0;
  int32_t nqb = 0, nkb = 0, npq = 0, npk = 0;
  int32_t gq = 1, gkv = 1, rq = 1, rkv = 1;
  int64_t Rp = 0;
  int64_t tiles_bound = 0;
  // device
  int64_t* tile_ptr = nullptr;  // null for Direct (logical CSR is used)
  int32_t* tile_kv = nullptr;
  uint64_t* member = nullptr;
  int32_t* counts = nullptr;
  int64_t* scan_tmp = nullptr;
  Task* tasks = nullptr;
  int64_t* task_ptr = nullptr;  // split > 1: [Rp + 1], device task count at [Rp]
  int64_t tasks_bound = 0;
  int32_t* order = nullptr;     // dispatch order of the tasks (Split-K plans); null: as stored
  Task* tasks_run = nullptr;    // the tasks in dispatch order (plans without Split-K); null: row order
  int32_t* dispatch = nullptr;  // the dispatch order (exported); null: row order
  float* ws = nullptr;
  int64_t ws_bytes = 0;
  // split-free plans whose XCDs work in groups: the groups' shares of the
  // task list, cut to hold equal work, and the launch slots they need
  bool balanced = false;
  int32_t share_lo[5] = {0, 0, 0, 0, 0};
  int64_t nslots = 0;
};

}  // namespace

struct bsa_plan_s {
  int dev = 0;
  hipStream_t stream = nullptr;
  bsa_shapes shapes{};
  int32_t B = 0, H = 0, Nq = 0, Nkv = 0;
  std::vector<HeadDesc> heads;
  std::vector<int64_t> row_base;
  int64_t R = 0, nnz = 0;
  std::vector<void*> allocs;
  hipEvent_t ready = nullptr, done = nullptr;
  // device
  uint16_t* zero_page = nullptr;

  HeadDesc* heads_dev = nullptr;
  int64_t* row_base_dev = nullptr;
  int32_t* seg_heads_dev = nullptr;
  SegStats* stats_dev = nullptr;
  unsigned long long* bh_nnz_dev = nullptr;
  int32_t* counts_dev = nullptr;
  int64_t* row_ptr_dev = nullptr;
  int64_t* scan_tmp_dev = nullptr;
  int32_t* col_idx_dev = nullptr;
  std::vector<Segment> segs;

  ~bsa_plan_s() {
    if (done) (void)hipStreamWaitEvent(stream, done, 0);
    for (void* p : allocs) (void)hipFreeAsync(p, stream);
    if (ready) (void)hipEventDestroy(ready);
    if (done) (void)hipEventDestroy(done);
  }

  // Fault injection for tests: BSA_FAULT_ALLOC=n makes the n-th device
  // allocation of a plan fail (n >= 1), so that error paths that already
  // hold allocations can be checked for leaks.
  bsa_status alloc(void** p, size_t bytes) {
    *p = nullptr;
    if (const char* f = std::getenv("BSA_FAULT_ALLOC")) {
      const long n = std::atol(f);
      if (n >= 1 && (long)allocs.size() + 1 == n)
        return fail(BSA_ERR_OOM, "device allocation " + std::to_string(n) + " failed (injected by BSA_FAULT_ALLOC)");
    }
    if (bytes == 0) bytes = 256;
    hipError_t e = hipMallocAsync(p, bytes, stream);
    if (e != hipSuccess) {
      *p = nullptr;
      (void)hipGetLastError();
      return fail(e == hipErrorOutOfMemory ? BSA_ERR_OOM : BSA_ERR_HIP,
                  "device allocation of " + std::to_string(bytes) + " bytes failed: " + hipGetErrorString(e));
    }
    allocs.push_back(*p);
    return BSA_OK;
  }
};

namespace {

bsa_status validate_shapes(const bsa_shapes* s) {
  if (!s) return fail(BSA_ERR_INVALID, "shapes is NULL");
  if (s->batch < 1 || s->heads < 1 || s->seq_q < 1 || s->seq_kv < 1 || s->head_dim < 1)
    return fail(BSA_ERR_INVALID, "batch, heads, seq_q, seq_kv and head_dim must be positive");
  if (s->dtype != BSA_DTYPE_BF16 && s->dtype != BSA_DTYPE_F16 && s->dtype != BSA_DTYPE_F32)
    return fail(BSA_ERR_INVALID, "unknown dtype");
  const int64_t* strides[] = {s->q_stride, s->k_stride, s->v_stride, s->o_stride};
  for (const int64_t* st : strides)
    for (int i = 0; i < 3; ++i)
      if (st[i] < 0) return fail(BSA_ERR_INVALID, "negative stride");
  return BSA_OK;
}

bsa_status select_segment_plan(Segment& sg, const bsa_shapes& s, const bsa_plan_opts& opts, const Lut* lut) {
  if (opts.force_plan >= 0) {
    const CatalogEntry* e = catalog_find(opts.force_plan);
    if (!e) return fail(BSA_ERR_INVALID, "force_plan names no catalog plan");
    if (const char* why = ineligible_reason(*e, sg.bq, sg.bkv, s))
      return fail(BSA_ERR_UNSUPPORTED, std::string("forced plan is not eligible: ") + why);
    sg.plan = *e;
    sg.regime_hit = false;
    return BSA_OK;
  }
  bsa_regime_query z{};
  z.bq = sg.bq;
  z.bkv = sg.bkv;
  z.dtype = s.dtype;
  z.head_dim = s.head_dim;
  z.batch_heads = (int64_t)s.batch * (int64_t)sg.heads.size();
  z.seq_q = s.seq_q;
  z.seq_kv = s.seq_kv;
  z.nnz = sg.nnz;
  z.blocks = sg.blocks;
  z.run_blocks = sg.run_blocks;
  z.max_row_nnz = sg.max_row_nnz;
  bool hit = false;
  std::vector<int32_t> ranking;
  if (opts.select_mode == 1) {
    const int32_t b = base_plan(sg.bq, sg.bkv);
    if (b >= 0) ranking.push_back(b);
  } else {
    ranking = lut_ranking(lut, z, &hit);
  }
  std::string why_all;
  for (int32_t id : ranking) {
    const CatalogEntry* e = catalog_find(id);
    if (!e) continue;
    const char* why = ineligible_reason(*e, sg.bq, sg.bkv, s);
    if (!why) {
      sg.plan = *e;
      sg.regime_hit = hit;
      if (log_on())
        std::fprintf(stderr, "[bsa] segment B=(%d,%d): regime %s, plan %d (T=(%d,%d), split %d)\n", sg.bq, sg.bkv,
                     hit ? "hit" : "miss", e->id, e->tq, e->tkv, e->split);
      return BSA_OK;
    }
    why_all += std::string(" plan ") + std::to_string(id) + ": " + why + ";";
  }
  return fail(BSA_ERR_UNSUPPORTED, "no-eligible-plan for B=(" + std::to_string(sg.bq) + "," +
                                       std::to_string(sg.bkv) + ")" + why_all);
}

}  // namespace

namespace {
// Every logical mask row starts on a 4-byte boundary and spans whole words,
// so the mask kernels may read rows as 32-bit words.
bool mask_rows_word_aligned(const bsa_mask* mask, const std::vector<HeadDesc>& heads) {
  if ((reinterpret_cast<uintptr_t>(mask->data) & 3) != 0 || (mask->stride_b & 3) != 0) return false;
  for (const HeadDesc& hd : heads)
    if ((hd.mask_off & 3) != 0 || (hd.nkb & 3) != 0) return false;
  return true;
}

bsa_status read_device_i64(bsa_plan_t plan, const int64_t* src, int64_t* dst) {
  HIP_TRY(hipMemcpyAsync(dst, src, sizeof(int64_t), hipMemcpyDeviceToHost, plan->stream));
  HIP_TRY(hipStreamSynchronize(plan->stream));
  return BSA_OK;
}

// Logical rows (global block-CSR row ids) of a Direct segment, in segment order.
std::vector<int64_t> segment_logical_rows(bsa_plan_t plan, const Segment& sg) {
  std::vector<int64_t> rows;
  rows.reserve((size_t)sg.Rp);
  for (int32_t b = 0; b < plan->B; ++b)
    for (int32_t h : sg.heads)
      for (int32_t pq = 0; pq < sg.npq; ++pq) rows.push_back(plan->row_base[(size_t)b * plan->H + h] + pq);
  return rows;
}
}  // namespace

extern "C" {

bsa_status bsa_version(int32_t* major, int32_t* minor) {
  if (!major || !minor) return fail(BSA_ERR_INVALID, "null output");
  *major = BSA_VERSION_MAJOR;
  *minor = BSA_VERSION_MINOR;
  return BSA_OK;
}

const char* bsa_status_string(bsa_status s) {
  switch (s) {
    case BSA_OK: return "ok";
    case BSA_ERR_INVALID: return "invalid argument";
    case BSA_ERR_UNSUPPORTED: return "no eligible plan";
    case BSA_ERR_HIP: return "HIP error";
    case BSA_ERR_OOM: return "out of memory";
    case BSA_ERR_LUT: return "plan table error";
  }
  return "unknown status";
}

const char* bsa_last_error(void) { return g_err.c_str(); }

bsa_status bsa_lut_load(const char* path, bsa_lut_t* out) {
  if (!out) return fail(BSA_ERR_INVALID, "out is NULL");
  *out = nullptr;
  if (!path) return fail(BSA_ERR_INVALID, "path is NULL");
  std::string text, err;
  if (!read_file(path, &text)) return fail(BSA_ERR_LUT, std::string("cannot read ") + path);
  std::unique_ptr<bsa_lut_s> l(new (std::nothrow) bsa_lut_s());
  if (!l) return fail(BSA_ERR_OOM, "host allocation failed");
  if (!lut_parse(text, &l->lut, &err)) return fail(BSA_ERR_LUT, std::string(path) + ": " + err);
  *out = l.release();
  return BSA_OK;
}

bsa_status bsa_lut_destroy(bsa_lut_t lut) {
  delete lut;
  return BSA_OK;
}

bsa_status bsa_lut_rank(bsa_lut_t lut, const bsa_regime_query* z, int32_t* plans, int32_t cap, int32_t* n,
                        int32_t* hit) {
  if (!z || !n || (cap > 0 && !plans) || cap < 0) return fail(BSA_ERR_INVALID, "bad arguments");
  bool h = false;
  const Lut* l = lut ? &lut->lut : default_lut();
  std::vector<int32_t> r = lut_ranking(l, *z, &h);
  *n = (int32_t)r.size();
  if (hit) *hit = h ? 1 : 0;
  for (int32_t i = 0; i < cap && i < (int32_t)r.size(); ++i) plans[i] = r[i];
  return BSA_OK;
}

bsa_status bsa_select_plan(bsa_lut_t lut, const bsa_regime_query* z, const bsa_shapes* shapes, int32_t* plan_id) {
  if (!z || !shapes || !plan_id) return fail(BSA_ERR_INVALID, "bad arguments");
  *plan_id = -1;
  bsa_status st = validate_shapes(shapes);
  if (st != BSA_OK) return st;
  bool h = false;
  const Lut* l = lut ? &lut->lut : default_lut();
  for (int32_t id : lut_ranking(l, *z, &h)) {
    const CatalogEntry* e = catalog_find(id);
    if (e && !ineligible_reason(*e, z->bq, z->bkv, *shapes)) {
      *plan_id = id;
      return BSA_OK;
    }
  }
  return fail(BSA_ERR_UNSUPPORTED, "no-eligible-plan");
}

int32_t bsa_catalog_size(void) { return (int32_t)catalog().size(); }

bsa_status bsa_catalog_get(int32_t id, bsa_catalog_entry* out) {
  const CatalogEntry* e = catalog_find(id);
  if (!e || !out) return fail(BSA_ERR_INVALID, "bad catalog id or null output");
  *out = bsa_catalog_entry{e->id, e->tq, e->tkv, e->split, e->stages, e->waves, e->xcd_group};
  return BSA_OK;
}

bsa_status bsa_plan_eligible(int32_t plan_id, int32_t bq, int32_t bkv, const bsa_shapes* shapes,
                             int32_t* eligible) {
  const CatalogEntry* e = catalog_find(plan_id);
  if (!e || !shapes || !eligible || bq < 1 || bkv < 1) return fail(BSA_ERR_INVALID, "bad arguments");
  const char* why = ineligible_reason(*e, bq, bkv, *shapes);
  *eligible = why ? 0 : 1;
  if (why) g_err = why;
  return BSA_OK;
}

bsa_status bsa_base_plan(int32_t bq, int32_t bkv, int32_t* plan_id) {
  if (!plan_id || bq < 1 || bkv < 1) return fail(BSA_ERR_INVALID, "bad arguments");
  *plan_id = base_plan(bq, bkv);
  if (*plan_id < 0) return fail(BSA_ERR_UNSUPPORTED, "no catalog tile nests with this geometry");
  return BSA_OK;
}

bsa_status bsa_plan(const bsa_mask* mask, const int32_t* B_Q, const int32_t* B_KV, int32_t n_geom,
                    const bsa_shapes* shapes, const bsa_plan_opts* opts_in, void* stream_in, bsa_plan_t* out) {
  if (!out) return fail(BSA_ERR_INVALID, "out is NULL");
  *out = nullptr;
  bsa_status st = validate_shapes(shapes);
  if (st != BSA_OK) return st;
  if (!mask || !mask->data) return fail(BSA_ERR_INVALID, "mask or mask data is NULL");
  if (mask->stride_b < 0) return fail(BSA_ERR_INVALID, "negative mask batch stride");
  if (!B_Q || !B_KV) return fail(BSA_ERR_INVALID, "block geometry is NULL");
  const bsa_shapes s = *shapes;
  if (n_geom != 1 && n_geom != s.heads) return fail(BSA_ERR_INVALID, "n_geom must be 1 or heads");
  for (int32_t i = 0; i < n_geom; ++i)
    if (B_Q[i] < 1 || B_KV[i] < 1 || B_Q[i] > 65536 || B_KV[i] > 65536)
      return fail(BSA_ERR_INVALID, "block sizes must lie in [1, 65536]");
  bsa_plan_opts opts{};
  opts.force_plan = -1;
  if (opts_in) opts = *opts_in;
  if (const char* fp = std::getenv("BSA_FORCE_PLAN")) {
    if (!opts_in || opts_in->force_plan < 0) opts.force_plan = std::atoi(fp);
  }
  const Lut* lut = opts.lut ? &opts.lut->lut : default_lut();
  hipStream_t stream = (hipStream_t)stream_in;

  std::unique_ptr<bsa_plan_s> p(new (std::nothrow) bsa_plan_s());
  if (!p) return fail(BSA_ERR_OOM, "host allocation failed");
  HIP_TRY(hipGetDevice(&p->dev));
  prepare_pool(p->dev);
  p->stream = stream;
  p->shapes = s;
  p->B = s.batch;
  p->H = s.heads;
  p->Nq = s.seq_q;
  p->Nkv = s.seq_kv;
  HIP_TRY(hipEventCreateWithFlags(&p->ready, hipEventDisableTiming));
  HIP_TRY(hipEventCreateWithFlags(&p->done, hipEventDisableTiming));

  // ---- per-head geometry, segments, logical row bases
  const int32_t H = s.heads, B = s.batch;
  std::map<std::pair<int32_t, int32_t>, int32_t> seg_of;
  p->heads.resize(H);
  bool uniform = true;
  for (int32_t h = 0; h < H; ++h) {
    const int32_t bq = B_Q[n_geom == 1 ? 0 : h], bkv = B_KV[n_geom == 1 ? 0 : h];
    if (bq != B_Q[0] || bkv != B_KV[0]) uniform = false;
    auto key = std::make_pair(bq, bkv);
    auto it = seg_of.find(key);
    if (it == seg_of.end()) {
      if ((int)p->segs.size() >= BSA_MAX_SEGMENTS) return fail(BSA_ERR_INVALID, "too many distinct block geometries");
      it = seg_of.emplace(key, (int32_t)p->segs.size()).first;
      p->segs.emplace_back();
      p->segs.back().bq = bq;
      p->segs.back().bkv = bkv;
    }
    Segment& sg = p->segs[it->second];
    sg.heads.push_back(h);
    HeadDesc& hd = p->heads[h];
    hd.nqb = (int32_t)cdiv(s.seq_q, bq);
    hd.nkb = (int32_t)cdiv(s.seq_kv, bkv);
    hd.seg = it->second;
    hd.pad = 0;
    sg.nqb = hd.nqb;
    sg.nkb = hd.nkb;
  }
  if (!mask->head_offset && !uniform)
    return fail(BSA_ERR_INVALID, "per-head geometries need mask head offsets");
  for (int32_t h = 0; h < H; ++h) {
    const int64_t sz = (int64_t)p->heads[h].nqb * p->heads[h].nkb;
    p->heads[h].mask_off = mask->head_offset ? mask->head_offset[h] : (int64_t)h * sz;
    if (p->heads[h].mask_off < 0) return fail(BSA_ERR_INVALID, "negative mask head offset");
  }
  p->row_base.assign((size_t)B * H + 1, 0);
  for (int32_t b = 0; b < B; ++b)
    for (int32_t h = 0; h < H; ++h)
      p->row_base[(size_t)b * H + h + 1] = p->row_base[(size_t)b * H + h] + p->heads[h].nqb;
  p->R = p->row_base.back();
  if (p->R >= INT32_MAX) return fail(BSA_ERR_UNSUPPORTED, "too many logical block rows");
  std::vector<int32_t> seg_heads;
  for (Segment& sg : p->segs) {
    sg.seg_heads_off = (int32_t)seg_heads.size();
    seg_heads.insert(seg_heads.end(), sg.heads.begin(), sg.heads.end());
  }
  const int nseg = (int)p->segs.size();

  // row chunks for the statistics reduction: within one (b, h), at most 2048 rows each
  std::vector<RowChunk> chunks;
  for (int b = 0; b < B; ++b)
    for (int h = 0; h < H; ++h) {
      const int bh = b * H + h;
      for (int64_t r = p->row_base[bh]; r < p->row_base[bh + 1]; r += 2048)
        chunks.push_back(RowChunk{r, std::min<int64_t>(r + 2048, p->row_base[bh + 1]), bh, p->heads[h].seg});
    }

  // ---- device buffer before the statistics synchronisation
  const size_t o_zero = 0;
  const size_t o_heads = align256(o_zero + 256);
  const size_t o_rbase = align256(o_heads + sizeof(HeadDesc) * H);
  const size_t o_sheads = align256(o_rbase + sizeof(int64_t) * p->row_base.size());
  const size_t o_stats = align256(o_sheads + sizeof(int32_t) * seg_heads.size());
  const size_t o_bhnnz = align256(o_stats + sizeof(SegStats) * nseg);
  const size_t o_chunks = align256(o_bhnnz + sizeof(unsigned long long) * (size_t)B * H);
  const size_t upload_bytes = o_chunks + sizeof(RowChunk) * chunks.size();
  const size_t o_counts = align256(upload_bytes);
  const size_t o_runs = align256(o_counts + sizeof(int32_t) * (size_t)p->R);
  const size_t o_rowptr = align256(o_runs + sizeof(int32_t) * (size_t)p->R);
  const size_t o_scan = align256(o_rowptr + sizeof(int64_t) * (size_t)(p->R + 1));
  const size_t pre_bytes = o_scan + sizeof(int64_t) * (size_t)scan_tmp_elems(p->R);
  void* pre = nullptr;
  if ((st = p->alloc(&pre, pre_bytes)) != BSA_OK) return st;
  uint8_t* pre8 = static_cast<uint8_t*>(pre);
  p->zero_page = reinterpret_cast<uint16_t*>(pre8 + o_zero);
  p->heads_dev = reinterpret_cast<HeadDesc*>(pre8 + o_heads);
  p->row_base_dev = reinterpret_cast<int64_t*>(pre8 + o_rbase);
  p->seg_heads_dev = reinterpret_cast<int32_t*>(pre8 + o_sheads);
  p->stats_dev = reinterpret_cast<SegStats*>(pre8 + o_stats);
  p->bh_nnz_dev = reinterpret_cast<unsigned long long*>(pre8 + o_bhnnz);
  p->counts_dev = reinterpret_cast<int32_t*>(pre8 + o_counts);
  p->row_ptr_dev = reinterpret_cast<int64_t*>(pre8 + o_rowptr);
  p->scan_tmp_dev = reinterpret_cast<int64_t*>(pre8 + o_scan);

  std::vector<SegStats> stats(nseg);
  std::vector<unsigned long long> bh_nnz;
  {
    Staging& stg = staging();
    std::lock_guard<std::mutex> lk(stg.mu);
    const size_t stats_at = align256(upload_bytes);
    const size_t bhnnz_at = align256(stats_at + sizeof(SegStats) * nseg);
    if (bhnnz_at - stats_at != o_bhnnz - o_stats) return fail(BSA_ERR_HIP, "statistics staging layout");
    if ((st = stg.reserve(bhnnz_at + sizeof(unsigned long long) * (size_t)B * H)) != BSA_OK) return st;
    uint8_t* h8 = static_cast<uint8_t*>(stg.ptr);
    std::memset(h8, 0, upload_bytes);
    std::memcpy(h8 + o_heads, p->heads.data(), sizeof(HeadDesc) * H);
    std::memcpy(h8 + o_rbase, p->row_base.data(), sizeof(int64_t) * p->row_base.size());
    std::memcpy(h8 + o_sheads, seg_heads.data(), sizeof(int32_t) * seg_heads.size());
    if (!chunks.empty()) std::memcpy(h8 + o_chunks, chunks.data(), sizeof(RowChunk) * chunks.size());
    HIP_TRY(hipMemcpyAsync(pre8, h8, upload_bytes, hipMemcpyHostToDevice, stream));

    // mu(M): row counts and statistics, then the block-CSR offsets
    MaskStateArgs ma{};
    ma.wide = mask_rows_word_aligned(mask, p->heads) ? 1 : 0;
    ma.mask = mask->data;
    ma.stride_b = mask->stride_b;
    ma.heads = p->heads_dev;
    ma.row_base = p->row_base_dev;
    ma.H = H;
    ma.nbh = B * H;
    ma.R = p->R;
    ma.counts = p->counts_dev;
    ma.runs = reinterpret_cast<int32_t*>(pre8 + o_runs);
    ma.chunks = reinterpret_cast<const RowChunk*>(pre8 + o_chunks);
    ma.nchunks = (int32_t)chunks.size();
    ma.seg_stats = p->stats_dev;
    ma.bh_nnz = p->bh_nnz_dev;
    HIP_TRY(launch_mask_count(ma, stream));
    HIP_TRY(launch_scan_i32(p->counts_dev, p->row_ptr_dev, p->R, p->scan_tmp_dev, stream));
    // the request's single synchronisation: the segment statistics and the
    // per-(b, h) active block counts
    // (one copy: both buffers start 256-aligned and lie at the same distance
    // apart on the device and in the staging buffer)
    static_assert(sizeof(SegStats) % 8 == 0, "statistics layout");
    HIP_TRY(hipMemcpyAsync(h8 + stats_at, p->stats_dev, (o_bhnnz - o_stats) + sizeof(unsigned long long) * (size_t)B * H,
                           hipMemcpyDeviceToHost, stream));
    HIP_TRY(hipStreamSynchronize(stream));
    std::memcpy(stats.data(), h8 + stats_at, sizeof(SegStats) * nseg);
    bh_nnz.resize((size_t)B * H);
    std::memcpy(bh_nnz.data(), h8 + bhnnz_at, sizeof(unsigned long long) * (size_t)B * H);
  }

  // ---- regime lookup and ranked fallback per segment (host)
  for (int k = 0; k < nseg; ++k) {
    Segment& sg = p->segs[k];
    sg.nnz = (int64_t)stats[k].nnz;
    sg.run_blocks = (int64_t)stats[k].run_blocks;
    sg.max_row_nnz = (int64_t)stats[k].max_row_nnz;
    sg.blocks = (int64_t)B * (int64_t)sg.heads.size() * sg.nqb * sg.nkb;
    p->nnz += sg.nnz;
    if ((st = select_segment_plan(sg, s, opts, lut)) != BSA_OK) return st;
    const CatalogEntry& e = sg.plan;
    sg.mapping = mapping_kind(sg.bq, sg.bkv, e.tq, e.tkv);
    sg.gq = e.tq >= sg.bq ? e.tq / sg.bq : 1;
    sg.gkv = e.tkv >= sg.bkv ? e.tkv / sg.bkv : 1;
    sg.rq = e.tq < sg.bq ? sg.bq / e.tq : 1;
    sg.rkv = e.tkv < sg.bkv ? sg.bkv / e.tkv : 1;
    sg.npq = (int32_t)cdiv(s.seq_q, e.tq);
    sg.npk = (int32_t)cdiv(s.seq_kv, e.tkv);
    sg.Rp = (int64_t)B * (int64_t)sg.heads.size() * sg.npq;
    sg.tiles_bound = sg.mapping == 0 ? sg.nnz : sg.nnz * sg.rq * sg.rkv;
    if (sg.tiles_bound >= INT32_MAX || sg.Rp >= INT32_MAX)
      return fail(BSA_ERR_UNSUPPORTED, "too many active tiles for 32-bit tile indices");
    sg.tasks_bound = e.split == 1 ? sg.Rp : std::min(sg.Rp * e.split, sg.Rp + sg.tiles_bound);
    if (sg.tasks_bound >= INT32_MAX) return fail(BSA_ERR_UNSUPPORTED, "too many tasks for one launch");
    sg.balanced = e.split == 1 && (e.xcd_group == 2 || e.xcd_group == 4);
    if (sg.balanced) {
      std::vector<int64_t> work;
      for (int b = 0; b < B; ++b)
        for (int32_t h : sg.heads) work.push_back((int64_t)bh_nnz[(size_t)b * H + h]);
      balanced_shares(work, sg.npq, e.xcd_group, sg.share_lo);
      sg.nslots = shares_slots(sg.share_lo, e.xcd_group, kSlotRun);
    }
  }
  if (p->nnz >= INT32_MAX) return fail(BSA_ERR_UNSUPPORTED, "too many active blocks");

  // ---- launch preparation of the selected plans only
  void* cptr = nullptr;
  if ((st = p->alloc(&cptr, sizeof(int32_t) * (size_t)p->nnz)) != BSA_OK) return st;
  p->col_idx_dev = static_cast<int32_t*>(cptr);
  {
    MaskStateArgs ma{};
    ma.mask = mask->data;
    ma.stride_b = mask->stride_b;
    ma.heads = p->heads_dev;
    ma.row_base = p->row_base_dev;
    ma.H = H;
    ma.nbh = B * H;
    ma.R = p->R;
    ma.row_ptr = p->row_ptr_dev;
    ma.col_idx = p->col_idx_dev;
    ma.wide = mask_rows_word_aligned(mask, p->heads) ? 1 : 0;
    HIP_TRY(launch_mask_fill(ma, stream));
  }
  for (Segment& sg : p->segs) {
    const CatalogEntry& e = sg.plan;
    const bool coarse = sg.gq * sg.gkv > 1;
    // sizes
    size_t need = 0;
    auto take = [&](size_t bytes) { size_t at = need; need = align256(need + bytes); return at; };
    const bool direct = sg.mapping == 0;
    const size_t o_counts2 = take(sizeof(int32_t) * (size_t)sg.Rp);
    const size_t o_scan2 = take(sizeof(int64_t) * (size_t)scan_tmp_elems(sg.Rp));
    const size_t o_tptr = direct ? 0 : take(sizeof(int64_t) * (size_t)(sg.Rp + 1));
    const size_t o_tkv = direct ? 0 : take(sizeof(int32_t) * (size_t)sg.tiles_bound);
    const size_t o_mem = (direct || !coarse) ? 0 : take(sizeof(uint64_t) * (size_t)sg.tiles_bound);
    const size_t o_tasks = take(sizeof(Task) * (size_t)sg.tasks_bound);
    const size_t o_taskptr = e.split > 1 ? take(sizeof(int64_t) * (size_t)(sg.Rp + 1)) : 0;
    // dispatch order: tasks with equal KV lists side by side.  Up to 512
    // tasks (two workgroups on each of 256 CUs) run all at once, so their
    // order does not change what shares an L2.
    const bool ordered = !opts.keep_row_order && sg.tasks_bound > kOrderMinTasks;
    size_t order_temp = 0;
    if (ordered) HIP_TRY(task_order_temp_bytes(sg.tasks_bound, &order_temp));
    const size_t nb = ordered ? (size_t)sg.tasks_bound : 0;
    const int64_t table_size = ordered ? task_order_table_size(sg.tasks_bound) : 0;
    const size_t o_tkey = take(sizeof(uint64_t) * (size_t)table_size), o_tmin = take(sizeof(int32_t) * (size_t)table_size);
    const size_t o_slot = take(sizeof(int32_t) * nb), o_iin = take(sizeof(int32_t) * nb);
    const size_t o_rep = take(sizeof(uint32_t) * nb), o_rsort = take(sizeof(uint32_t) * nb);
    const size_t o_order = take(sizeof(int32_t) * nb);
    const size_t o_otemp = take(order_temp);
    const size_t o_trun = take(e.split == 1 ? sizeof(Task) * nb : 0);
    void* buf = nullptr;
    if ((st = p->alloc(&buf, need)) != BSA_OK) return st;
    uint8_t* b8 = static_cast<uint8_t*>(buf);
    sg.counts = reinterpret_cast<int32_t*>(b8 + o_counts2);
    sg.scan_tmp = reinterpret_cast<int64_t*>(b8 + o_scan2);
    sg.tasks = reinterpret_cast<Task*>(b8 + o_tasks);
    if (direct) {
      sg.tile_ptr = nullptr;
      sg.tile_kv = p->col_idx_dev;
      sg.member = nullptr;
    } else {
      sg.tile_ptr = reinterpret_cast<int64_t*>(b8 + o_tptr);
      sg.tile_kv = reinterpret_cast<int32_t*>(b8 + o_tkv);
      sg.member = coarse ? reinterpret_cast<uint64_t*>(b8 + o_mem) : nullptr;
      MapArgs m{};
      m.mask = mask->data;
      m.stride_b = mask->stride_b;
      m.heads = p->heads_dev;
      m.seg_heads = p->seg_heads_dev + sg.seg_heads_off;
      m.nsh = (int32_t)sg.heads.size();
      m.H = H;
      m.npq = sg.npq;
      m.npk = sg.npk;
      m.nqb = sg.nqb;
      m.nkb = sg.nkb;
      m.gq = sg.gq;
      m.gkv = sg.gkv;
      m.rq = sg.rq;
      m.rkv = sg.rkv;
      m.Rp = sg.Rp;
      m.counts = sg.counts;
      m.wide = mask_rows_word_aligned(mask, p->heads) ? 1 : 0;
      HIP_TRY(launch_map_count(m, stream));
      HIP_TRY(launch_scan_i32(sg.counts, sg.tile_ptr, sg.Rp, sg.scan_tmp, stream));
      m.tile_ptr = sg.tile_ptr;
      m.tile_kv = sg.tile_kv;
      m.member = sg.member;
      HIP_TRY(launch_map_fill(m, stream));
    }
    TaskArgs ta{};
    ta.tile_ptr = direct ? p->row_ptr_dev : sg.tile_ptr;
    ta.row_base = p->row_base_dev;
    ta.seg_heads = p->seg_heads_dev + sg.seg_heads_off;
    ta.nsh = (int32_t)sg.heads.size();
    ta.H = H;
    ta.npq = sg.npq;
    ta.split = e.split;
    ta.direct = direct ? 1 : 0;
    ta.Rp = sg.Rp;
    ta.tasks = sg.tasks;
    if (e.split > 1) {
      sg.task_ptr = reinterpret_cast<int64_t*>(b8 + o_taskptr);
      ta.counts = sg.counts;
      HIP_TRY(launch_task_count(ta, stream));
      HIP_TRY(launch_scan_i32(sg.counts, sg.task_ptr, sg.Rp, sg.scan_tmp, stream));
      ta.task_ptr = sg.task_ptr;
      sg.ws_bytes = (int64_t)sizeof(float) * sg.tasks_bound * e.tq * (kHeadDim + 2);
      void* ws = nullptr;
      if ((st = p->alloc(&ws, (size_t)sg.ws_bytes)) != BSA_OK) return st;
      sg.ws = static_cast<float*>(ws);
    }
    HIP_TRY(launch_task_fill(ta, stream));
    if (ordered) {
      OrderArgs oa{};
      oa.tasks = sg.tasks;
      oa.ntasks_dev = e.split > 1 ? sg.task_ptr + sg.Rp : nullptr;
      oa.ntasks = sg.tasks_bound;
      oa.tile_kv = sg.tile_kv;
      oa.member = sg.member;
      oa.table_key = reinterpret_cast<uint64_t*>(b8 + o_tkey);
      oa.table_min = reinterpret_cast<int32_t*>(b8 + o_tmin);
      oa.table_size = table_size;
      oa.task_slot = reinterpret_cast<int32_t*>(b8 + o_slot);
      oa.idx_in = reinterpret_cast<int32_t*>(b8 + o_iin);
      oa.rep = reinterpret_cast<uint32_t*>(b8 + o_rep);
      oa.rep_sorted = reinterpret_cast<uint32_t*>(b8 + o_rsort);
      oa.order = reinterpret_cast<int32_t*>(b8 + o_order);
      oa.temp = b8 + o_otemp;
      oa.temp_bytes = order_temp;
      oa.tasks_out = e.split == 1 ? reinterpret_cast<Task*>(b8 + o_trun) : nullptr;
      HIP_TRY(launch_task_order(oa, stream));
      // without Split-K the kernel reads the reordered copy directly; the
      // row-order list stays for the plan export
      sg.tasks_run = oa.tasks_out;
      sg.order = e.split == 1 ? nullptr : oa.order;
      sg.dispatch = oa.order;
    }
  }
  HIP_TRY(hipEventRecord(p->ready, stream));
  *out = p.release();
  return BSA_OK;
}

bsa_status bsa_forward(bsa_plan_t plan, const void* q, const void* k, const void* v, void* o, float* lse,
                       void* stream_in) {
  if (!plan) return fail(BSA_ERR_INVALID, "plan is NULL");
  if (!q || !k || !v || !o) return fail(BSA_ERR_INVALID, "q, k, v and o must be device pointers");
  const uintptr_t mis = (reinterpret_cast<uintptr_t>(q) | reinterpret_cast<uintptr_t>(k) |
                         reinterpret_cast<uintptr_t>(v) | reinterpret_cast<uintptr_t>(o)) & 15;
  if (mis) return fail(BSA_ERR_INVALID, "q, k, v and o must be 16-byte aligned");
  if (lse && (reinterpret_cast<uintptr_t>(lse) & 3)) return fail(BSA_ERR_INVALID, "lse must be 4-byte aligned");
  hipStream_t stream = (hipStream_t)stream_in;
  HIP_TRY(hipStreamWaitEvent(stream, plan->ready, 0));
  const bsa_shapes& s = plan->shapes;
  for (const Segment& sg : plan->segs) {
    const CatalogEntry& e = sg.plan;
    AttnArgs a{};
    a.tasks = sg.tasks_run ? sg.tasks_run : sg.tasks;
    a.ntasks = (int32_t)sg.tasks_bound;
    a.ntasks_dev = e.split > 1 ? sg.task_ptr + sg.Rp : nullptr;
    a.order = sg.order;
    a.kv_tile = sg.tile_kv;
    a.member = sg.member;
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k);
    a.v = static_cast<const uint16_t*>(v);
    a.o = static_cast<uint16_t*>(o);
    a.lse = lse;
    a.ws = sg.ws;
    a.zero_page = plan->zero_page;
    a.qs0 = s.q_stride[0]; a.qs1 = s.q_stride[1]; a.qs2 = s.q_stride[2];
    a.ks0 = s.k_stride[0]; a.ks1 = s.k_stride[1]; a.ks2 = s.k_stride[2];
    a.vs0 = s.v_stride[0]; a.vs1 = s.v_stride[1]; a.vs2 = s.v_stride[2];
    a.os0 = s.o_stride[0]; a.os1 = s.o_stride[1]; a.os2 = s.o_stride[2];
    a.H = s.heads;
    a.Nq = s.seq_q;
    a.Nkv = s.seq_kv;
    a.bq_shift = sg.gq > 1 ? ilog2_exact(sg.bq) : 0;
    a.bkv_shift = sg.gkv > 1 ? ilog2_exact(sg.bkv) : 0;
    a.gq = sg.gq;
    a.gkv = sg.gkv;
    a.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)s.head_dim));
    a.slot_group = e.xcd_group;
    a.slot_run = kSlotRun;
    a.balanced = sg.balanced ? 1 : 0;
    for (int g = 0; g < 5; ++g) a.share_lo[g] = sg.share_lo[g];
    a.nslots = sg.nslots;
    HIP_TRY(launch_attention(e.tq, e.tkv, e.waves, e.stages, a, stream));
    if (e.split > 1) HIP_TRY(launch_splitk_merge(e.tq, a, stream));
  }
  HIP_TRY(hipEventRecord(plan->done, stream));
  return BSA_OK;
}

bsa_status bsa_plan_num_segments(bsa_plan_t plan, int32_t* n) {
  if (!plan || !n) return fail(BSA_ERR_INVALID, "bad arguments");
  *n = (int32_t)plan->segs.size();
  return BSA_OK;
}


bsa_status bsa_plan_info(bsa_plan_t plan, int32_t segment, bsa_segment_info* out) {
  if (!plan || !out || segment < 0 || segment >= (int32_t)plan->segs.size())
    return fail(BSA_ERR_INVALID, "bad arguments");
  const Segment& sg = plan->segs[segment];
  bsa_segment_info i{};
  i.bq = sg.bq;
  i.bkv = sg.bkv;
  i.n_heads = (int32_t)sg.heads.size();
  i.plan_id = sg.plan.id;
  i.tq = sg.plan.tq;
  i.tkv = sg.plan.tkv;
  i.split = sg.plan.split;
  i.mapping = sg.mapping;
  i.regime_hit = sg.regime_hit ? 1 : 0;
  i.nnz = sg.nnz;
  i.blocks = sg.blocks;
  i.run_blocks = sg.run_blocks;
  i.max_row_nnz = sg.max_row_nnz;
  i.n_rows = sg.Rp;
  i.workspace_bytes = sg.ws_bytes;
  // exact tile and task counts live on the device
  bsa_status st;
  if (sg.mapping == 0) {
    i.n_tiles = sg.nnz;
  } else if ((st = read_device_i64(plan, sg.tile_ptr + sg.Rp, &i.n_tiles)) != BSA_OK) {
    return st;
  }
  if (sg.plan.split == 1) {
    i.n_tasks = sg.Rp;
  } else if ((st = read_device_i64(plan, sg.task_ptr + sg.Rp, &i.n_tasks)) != BSA_OK) {
    return st;
  }
  *out = i;
  return BSA_OK;
}

bsa_status bsa_plan_segment_heads(bsa_plan_t plan, int32_t segment, int32_t* heads, int32_t cap, int32_t* n) {
  if (!plan || !n || segment < 0 || segment >= (int32_t)plan->segs.size() || cap < 0 || (cap > 0 && !heads))
    return fail(BSA_ERR_INVALID, "bad arguments");
  const Segment& sg = plan->segs[segment];
  *n = (int32_t)sg.heads.size();
  for (int32_t i = 0; i < cap && i < *n; ++i) heads[i] = sg.heads[i];
  return BSA_OK;
}

bsa_status bsa_plan_export(bsa_plan_t plan, int32_t segment, int32_t what, void* host_buf, size_t bytes,
                           size_t* needed) {
  if (!plan || !needed) return fail(BSA_ERR_INVALID, "bad arguments");
  const bool per_segment = what >= BSA_EXPORT_TILE_PTR;
  if (per_segment && (segment < 0 || segment >= (int32_t)plan->segs.size()))
    return fail(BSA_ERR_INVALID, "bad segment");
  hipStream_t s = plan->stream;
  auto copy_out = [&](const void* src, size_t n) -> bsa_status {
    *needed = n;
    if (!host_buf) return BSA_OK;
    if (bytes < n) return fail(BSA_ERR_INVALID, "export buffer too small");
    if (n) HIP_TRY(hipMemcpyAsync(host_buf, src, n, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    return BSA_OK;
  };
  auto host_vec_i64 = [&](const int64_t* src, int64_t n, std::vector<int64_t>* v) -> bsa_status {
    v->resize((size_t)n);
    if (n) HIP_TRY(hipMemcpyAsync(v->data(), src, sizeof(int64_t) * n, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    return BSA_OK;
  };
  bsa_status st;
  switch (what) {
    case BSA_EXPORT_ROW_PTR: return copy_out(plan->row_ptr_dev, sizeof(int64_t) * (size_t)(plan->R + 1));
    case BSA_EXPORT_COL_IDX: return copy_out(plan->col_idx_dev, sizeof(int32_t) * (size_t)plan->nnz);
    case BSA_EXPORT_BH_NNZ:
      return copy_out(plan->bh_nnz_dev, sizeof(int64_t) * (size_t)plan->B * plan->H);
    default: break;
  }
  const Segment& sg = plan->segs[segment];
  // Direct segments read the logical block-CSR; export their rows rebased
  // onto the segment's own tile list.
  std::vector<int64_t> lrows, lptr, seg_ptr;
  if (sg.mapping == 0 && what != BSA_EXPORT_TILE_MEMBER) {
    lrows = segment_logical_rows(plan, sg);
    if ((st = host_vec_i64(plan->row_ptr_dev, plan->R + 1, &lptr)) != BSA_OK) return st;
    seg_ptr.assign(lrows.size() + 1, 0);
    for (size_t r = 0; r < lrows.size(); ++r)
      seg_ptr[r + 1] = seg_ptr[r] + (lptr[(size_t)lrows[r] + 1] - lptr[(size_t)lrows[r]]);
  }
  switch (what) {
    case BSA_EXPORT_TILE_PTR: {
      if (sg.mapping != 0) return copy_out(sg.tile_ptr, sizeof(int64_t) * (size_t)(sg.Rp + 1));
      *needed = sizeof(int64_t) * seg_ptr.size();
      if (host_buf) {
        if (bytes < *needed) return fail(BSA_ERR_INVALID, "export buffer too small");
        std::memcpy(host_buf, seg_ptr.data(), *needed);
      }
      return BSA_OK;
    }
    case BSA_EXPORT_TILE_KV: {
      if (sg.mapping != 0) {
        int64_t nt = 0;
        if ((st = read_device_i64(plan, sg.tile_ptr + sg.Rp, &nt)) != BSA_OK) return st;
        return copy_out(sg.tile_kv, sizeof(int32_t) * (size_t)nt);
      }
      *needed = sizeof(int32_t) * (size_t)seg_ptr.back();
      if (!host_buf) return BSA_OK;
      if (bytes < *needed) return fail(BSA_ERR_INVALID, "export buffer too small");
      int32_t* dst = static_cast<int32_t*>(host_buf);
      for (size_t r = 0; r < lrows.size(); ++r) {
        const int64_t lo = lptr[(size_t)lrows[r]], hi = lptr[(size_t)lrows[r] + 1];
        if (hi > lo)
          HIP_TRY(hipMemcpyAsync(dst + seg_ptr[r], plan->col_idx_dev + lo, sizeof(int32_t) * (hi - lo),
                                 hipMemcpyDeviceToHost, s));
      }
      HIP_TRY(hipStreamSynchronize(s));
      return BSA_OK;
    }
    case BSA_EXPORT_TILE_MEMBER: {
      if (!sg.member) return copy_out(nullptr, 0);
      int64_t nt = 0;
      if ((st = read_device_i64(plan, sg.tile_ptr + sg.Rp, &nt)) != BSA_OK) return st;
      return copy_out(sg.member, sizeof(uint64_t) * (size_t)nt);
    }
    case BSA_EXPORT_TASKS: {
      int64_t nt = sg.Rp;
      if (sg.plan.split > 1 && (st = read_device_i64(plan, sg.task_ptr + sg.Rp, &nt)) != BSA_OK) return st;
      *needed = sizeof(int64_t) * 6 * (size_t)nt;
      if (!host_buf) return BSA_OK;
      if (bytes < *needed) return fail(BSA_ERR_INVALID, "export buffer too small");
      std::vector<Task> t((size_t)nt);
      if (nt) HIP_TRY(hipMemcpyAsync(t.data(), sg.tasks, sizeof(Task) * nt, hipMemcpyDeviceToHost, s));
      HIP_TRY(hipStreamSynchronize(s));
      int64_t* dst = static_cast<int64_t*>(host_buf);
      std::vector<int32_t> slot_of_head((size_t)plan->H, -1);
      for (size_t j = 0; j < sg.heads.size(); ++j) slot_of_head[(size_t)sg.heads[j]] = (int32_t)j;
      for (int64_t i = 0; i < nt; ++i) {
        int64_t lo = t[i].tile_begin, hi = t[i].tile_end;
        if (sg.mapping == 0) {
          // rebase from the global block-CSR onto the segment's tile list
          const int64_t b = t[i].bh / plan->H, h = t[i].bh % plan->H;
          const int64_t rs = (b * (int64_t)sg.heads.size() + slot_of_head[(size_t)h]) * sg.npq + t[i].pq;
          const int64_t shift = seg_ptr[(size_t)rs] - lptr[(size_t)lrows[(size_t)rs]];
          lo += shift;
          hi += shift;
        }
        const int64_t f[6] = {t[i].bh, t[i].pq, lo, hi, t[i].split, t[i].nsplit};
        std::memcpy(dst + 6 * i, f, sizeof f);
      }
      return BSA_OK;
    }
    case BSA_EXPORT_DISPATCH: {
      int64_t nt = sg.Rp;
      if (sg.plan.split > 1 && (st = read_device_i64(plan, sg.task_ptr + sg.Rp, &nt)) != BSA_OK) return st;
      *needed = sizeof(int64_t) * (size_t)nt;
      if (!host_buf) return BSA_OK;
      if (bytes < *needed) return fail(BSA_ERR_INVALID, "export buffer too small");
      std::vector<int32_t> o((size_t)nt);
      if (sg.dispatch && nt) {
        HIP_TRY(hipMemcpyAsync(o.data(), sg.dispatch, sizeof(int32_t) * nt, hipMemcpyDeviceToHost, s));
        HIP_TRY(hipStreamSynchronize(s));
      } else {
        for (int64_t i = 0; i < nt; ++i) o[(size_t)i] = (int32_t)i;
      }
      int64_t* dst = static_cast<int64_t*>(host_buf);
      for (int64_t i = 0; i < nt; ++i) dst[i] = o[(size_t)i];
      return BSA_OK;
    }
    default: return fail(BSA_ERR_INVALID, "unknown export selector");
  }
}

bsa_status bsa_plan_destroy(bsa_plan_t plan) {
  delete plan;
  return BSA_OK;
}

namespace {

// Checks shared by both sparsifier entry points; fills the block grid.
bsa_status sparsify_validate(const void* q, const void* k, const bsa_shapes* shapes, int32_t bq, int32_t bkv,
                             uint8_t* mask, int64_t* nqb, int64_t* nkb) {
  if (!q || !k || !mask) return fail(BSA_ERR_INVALID, "q, k and mask must be device pointers");
  bsa_status st = validate_shapes(shapes);
  if (st != BSA_OK) return st;
  if (bq < 1 || bkv < 1) return fail(BSA_ERR_INVALID, "block sizes must be positive");
  const bsa_shapes& s = *shapes;
  if (s.dtype != BSA_DTYPE_BF16) return fail(BSA_ERR_UNSUPPORTED, "only bfloat16 tensors are implemented");
  if (s.head_dim != kHeadDim) return fail(BSA_ERR_UNSUPPORTED, "only head_dim 128 is implemented");
  *nqb = cdiv(s.seq_q, bq);
  *nkb = cdiv(s.seq_kv, bkv);
  if (*nkb > sparsify_max_kv_blocks())
    return fail(BSA_ERR_UNSUPPORTED, "more than " + std::to_string(sparsify_max_kv_blocks()) + " KV blocks per row");
  return BSA_OK;
}

// Device bytes of one head's block means (queries and keys) and score rows.
int64_t sparsify_head_bytes(int64_t nqb, int64_t nkb) {
  return (nqb + nkb) * kHeadDim * (int64_t)sizeof(double) + nqb * nkb * (int64_t)sizeof(double);
}

// The sparsifier's passes over the heads, `chunk` heads at a time, with the
// block means and score rows of a pass in `work` (at least chunk * head bytes).
hipError_t sparsify_passes(const void* q, const void* k, const bsa_shapes& s, int32_t bq, int32_t bkv, int32_t topk,
                           int32_t diagonal, uint8_t* mask, int64_t nqb, int64_t nkb, int64_t chunk, void* work,
                           hipStream_t stream) {
  const int64_t nbh = (int64_t)s.batch * s.heads;
  const size_t bytes_q = (size_t)(chunk * nqb * kHeadDim) * sizeof(double);
  const size_t bytes_k = (size_t)(chunk * nkb * kHeadDim) * sizeof(double);
  double* pq = static_cast<double*>(work);
  double* pk = reinterpret_cast<double*>(static_cast<uint8_t*>(work) + bytes_q);
  double* sc = reinterpret_cast<double*>(static_cast<uint8_t*>(work) + bytes_q + bytes_k);
  const uint16_t* qh = static_cast<const uint16_t*>(q);
  const uint16_t* kh = static_cast<const uint16_t*>(k);
  hipError_t e = hipSuccess;
  for (int64_t bh0 = 0; bh0 < nbh && e == hipSuccess; bh0 += chunk) {
    const int32_t n = (int32_t)std::min<int64_t>(chunk, nbh - bh0);
    e = launch_block_mean(qh, s.q_stride[0], s.q_stride[1], s.q_stride[2], s.heads, s.seq_q, bq, (int32_t)bh0, n, pq,
                          stream);
    if (e == hipSuccess)
      e = launch_block_mean(kh, s.k_stride[0], s.k_stride[1], s.k_stride[2], s.heads, s.seq_kv, bkv, (int32_t)bh0, n,
                            pk, stream);
    if (e == hipSuccess) e = launch_block_scores(pq, pk, (int32_t)nqb, (int32_t)nkb, n, sc, stream);
    if (e == hipSuccess)
      e = launch_topk_select(sc, (int32_t)nqb, (int32_t)nkb, topk, diagonal ? 1 : 0, s.seq_q, s.seq_kv, bq, bkv,
                             (int32_t)bh0, n, mask, stream);
  }
  return e;
}

// Scratch of the allocation-free sparsifier: one copy per device, resident
// until the process ends.  Host code never passes `scratch` itself to a
// kernel (in host code it names a host-side stand-in); it uses the device
// address that hipGetSymbolAddress returns for the current device.
constexpr int64_t kNoAllocScratchBytes = int64_t(64) << 20;
static __device__ __attribute__((aligned(256))) uint8_t scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on device `dev` (looked up once per device,
// with that device current).
bsa_status scratch_address(int dev, void** out) {
  *out = nullptr;
  if (dev < 0 || dev >= kMaxDevices) return fail(BSA_ERR_UNSUPPORTED, "device index beyond the scratch table");
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
      return fail(BSA_ERR_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return BSA_OK;
}

}  // namespace

bsa_status bsa_sparsify_topk(const void* q, const void* k, const bsa_shapes* shapes, int32_t bq, int32_t bkv,
                             int32_t topk, int32_t diagonal, uint8_t* mask, void* stream_in) {
  int64_t nqb = 0, nkb = 0;
  bsa_status st = sparsify_validate(q, k, shapes, bq, bkv, mask, &nqb, &nkb);
  if (st != BSA_OK) return st;
  const bsa_shapes& s = *shapes;
  hipStream_t stream = (hipStream_t)stream_in;
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  prepare_pool(dev);
  const int64_t nbh = (int64_t)s.batch * s.heads;
  // heads per pass: score rows of at most 256 MiB
  const int64_t per_scores = nqb * nkb * (int64_t)sizeof(double);
  const int64_t chunk = std::max<int64_t>(1, std::min<int64_t>(nbh, (int64_t(256) << 20) / per_scores));
  void* work = nullptr;
  HIP_TRY(hipMallocAsync(&work, (size_t)(chunk * sparsify_head_bytes(nqb, nkb)), stream));
  const hipError_t e = sparsify_passes(q, k, s, bq, bkv, topk, diagonal, mask, nqb, nkb, chunk, work, stream);
  const hipError_t ef = hipFreeAsync(work, stream);
  if (e != hipSuccess) return fail(BSA_ERR_HIP, std::string("sparsifier launch: ") + hipGetErrorString(e));
  if (ef != hipSuccess) return fail(BSA_ERR_HIP, std::string("hipFreeAsync: ") + hipGetErrorString(ef));
  return BSA_OK;
}

bsa_status bsa_sparsify_topk_noalloc(const void* q, const void* k, const bsa_shapes* shapes, int32_t bq,
                                     int32_t bkv, int32_t topk, int32_t diagonal, uint8_t* mask, void* stream_in) {
  int64_t nqb = 0, nkb = 0;
  bsa_status st = sparsify_validate(q, k, shapes, bq, bkv, mask, &nqb, &nkb);
  if (st != BSA_OK) return st;
  const int64_t per_head = sparsify_head_bytes(nqb, nkb);
  if (per_head > kNoAllocScratchBytes)
    return fail(BSA_ERR_INVALID, "one head needs " + std::to_string(per_head) +
                                     " bytes of block means and scores, more than the " +
                                     std::to_string(kNoAllocScratchBytes) + "-byte scratch of this entry point");
  const bsa_shapes& s = *shapes;
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  void* work = nullptr;
  if ((st = scratch_address(dev, &work)) != BSA_OK) return st;
  const int64_t nbh = (int64_t)s.batch * s.heads;
  const int64_t chunk = std::max<int64_t>(1, std::min<int64_t>(nbh, kNoAllocScratchBytes / per_head));
  // every byte of the scratch that a pass reads is written earlier in the
  // same pass (means before scores, scores before the selection), so nothing
  // needs clearing
  const hipError_t e =
      sparsify_passes(q, k, s, bq, bkv, topk, diagonal, mask, nqb, nkb, chunk, work, (hipStream_t)stream_in);
  if (e != hipSuccess) return fail(BSA_ERR_HIP, std::string("sparsifier launch: ") + hipGetErrorString(e));
  return BSA_OK;
}

}  // extern "C"
