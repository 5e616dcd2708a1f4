// Native catalog, Eligible(P, R), base plans, the plan-table artifact and the
// online lookup of Algorithm 2 (host code, no GPU calls).
#include "catalog.h"

#include <cctype>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <algorithm>

namespace bsa {

namespace {

// Ring depth and wavefronts of the kernel that runs tile (tq, tkv) with one
// wave per 32 query rows (64 rows per wave for (256, 32)).
int32_t default_stages(int tq, int tkv) { return (tq == 256 && tkv == 32) ? 8 : tkv == 32 ? 4 : 2; }
int32_t default_waves(int tq, int tkv) { return (tq == 256 && tkv == 32) ? 4 : tq / 32; }

std::vector<CatalogEntry> build_catalog() {
  const int tqs[] = {64, 128, 256};
  const int tkvs[] = {32, 64};
  const int splits[] = {1, 2, 4, 8};
  std::vector<CatalogEntry> out;
  int id = 0;
  // ids 0-23: ((tq index) * 2 + tkv index) * 4 + split index, XCD pairs
  for (int tq : tqs)
    for (int tkv : tkvs)
      for (int s : splits) out.push_back(CatalogEntry{id++, tq, tkv, s, default_stages(tq, tkv), default_waves(tq, tkv), 2});
  // ids 24-29: the split-free tiles with every XCD on the same stretch of tasks
  for (int tq : tqs)
    for (int tkv : tkvs) out.push_back(CatalogEntry{id++, tq, tkv, 1, default_stages(tq, tkv), default_waves(tq, tkv), 8});
  // ids 30-32: the other ring depth of three split-free tiles, XCD pairs.
  // (64, 32) with two slots fits four workgroups per CU (two waves per SIMD
  // instead of one, each load with one iteration to land instead of three);
  // (128, 32) with two slots (the same occupancy, a shallower prefetch);
  // (256, 64) with four slots (loads with three iterations to land).
  out.push_back(CatalogEntry{id++, 64, 32, 1, 2, 2, 2});
  out.push_back(CatalogEntry{id++, 128, 32, 1, 2, 4, 2});
  out.push_back(CatalogEntry{id++, 256, 64, 1, 4, 8, 2});
  // ids 33-34: the two-slot (64, 32) and (128, 32) with every XCD on the
  // same stretch of tasks
  out.push_back(CatalogEntry{id++, 64, 32, 1, 2, 2, 8});
  out.push_back(CatalogEntry{id++, 128, 32, 1, 2, 4, 8});
  return out;
}

}  // namespace

namespace {

bool nests(int32_t t, int32_t b) { return t > 0 && b > 0 && (t % b == 0 || b % t == 0); }

bool is_pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }

}  // namespace

const std::vector<CatalogEntry>& catalog() {
  static const std::vector<CatalogEntry> c = build_catalog();
  return c;
}

const CatalogEntry* catalog_find(int32_t id) {
  const auto& c = catalog();
  if (id < 0 || id >= (int32_t)c.size()) return nullptr;
  return &c[id];
}

int mapping_kind(int32_t bq, int32_t bkv, int32_t tq, int32_t tkv) {
  if (tq == bq && tkv == bkv) return 0;
  if (tq >= bq && tkv >= bkv) return 1;
  if (tq <= bq && tkv <= bkv) return 2;
  return 3;
}

const char* ineligible_reason(const CatalogEntry& e, int32_t bq, int32_t bkv, const bsa_shapes& s) {
  if (s.dtype != BSA_DTYPE_BF16) return "only bfloat16 tensors are implemented";
  if (s.head_dim != 128) return "only head_dim 128 is implemented";
  const int64_t* strides[] = {s.q_stride, s.k_stride, s.v_stride, s.o_stride};
  for (const int64_t* st : strides)
    for (int i = 0; i < 3; ++i)
      if (st[i] < 0 || st[i] % 8 != 0) return "strides must be non-negative multiples of 8 elements (16 bytes)";
  // the attention kernel addresses one head's K and V rows with 32-bit byte
  // offsets (up to a tile past the sequence end)
  const int64_t row_bytes = 2 * std::max(s.k_stride[2], s.v_stride[2]);
  if (((int64_t)s.seq_kv + 64) * row_bytes + 256 > 0xFFFFFFFFll)
    return "the K/V rows of one head must span less than 4 GiB";
  if (!nests(e.tq, bq)) return "query tile and query block do not nest";
  if (!nests(e.tkv, bkv)) return "KV tile and KV block do not nest";
  const int64_t gq = e.tq >= bq ? e.tq / bq : 1, gkv = e.tkv >= bkv ? e.tkv / bkv : 1;
  if (gq * gkv > 64) return "coarsened tile has more than 64 member blocks";
  if ((gq > 1 && !is_pow2(bq)) || (gkv > 1 && !is_pow2(bkv))) return "coarsened blocks must be powers of two";
  if (e.split < 1) return "bad split";
  return nullptr;
}

int32_t base_plan(int32_t bq, int32_t bkv) {
  bsa_shapes s{};
  s.head_dim = 128;
  s.dtype = BSA_DTYPE_BF16;
  int32_t best = -1;
  double best_dq = 0, best_dk = 0;
  for (const auto& e : catalog()) {
    if (e.split != 1 || ineligible_reason(e, bq, bkv, s)) continue;
    const double dq = std::fabs(std::log2((double)e.tq) - std::log2((double)bq));
    const double dk = std::fabs(std::log2((double)e.tkv) - std::log2((double)bkv));
    if (best < 0 || dq + dk < best_dq + best_dk || (dq + dk == best_dq + best_dk && dq < best_dq)) {
      best = e.id;
      best_dq = dq;
      best_dk = dk;
    }
  }
  return best;
}

// ---------------------------------------------------------------------------
// Minimal JSON reader for the artifact (objects, arrays, numbers, strings,
// true/false/null).

namespace {

struct JVal {
  enum Kind { kNull, kBool, kNum, kStr, kArr, kObj } kind = kNull;
  double num = 0;
  bool b = false;
  std::string str;
  std::vector<JVal> arr;
  std::vector<std::pair<std::string, JVal>> obj;
  const JVal* get(const char* key) const {
    for (const auto& kv : obj)
      if (kv.first == key) return &kv.second;
    return nullptr;
  }
};

struct JParser {
  const std::string& t;
  size_t i = 0;
  std::string err;
  explicit JParser(const std::string& text) : t(text) {}
  void ws() {
    while (i < t.size() && std::isspace((unsigned char)t[i])) ++i;
  }
  bool fail(const char* m) {
    if (err.empty()) err = std::string(m) + " at offset " + std::to_string(i);
    return false;
  }
  bool str(std::string* out) {
    if (t[i] != '"') return fail("expected string");
    ++i;
    out->clear();
    while (i < t.size() && t[i] != '"') {
      if (t[i] == '\\') {
        ++i;
        if (i >= t.size()) return fail("bad escape");
        char c = t[i];
        out->push_back(c == 'n' ? '\n' : c == 't' ? '\t' : c);
      } else {
        out->push_back(t[i]);
      }
      ++i;
    }
    if (i >= t.size()) return fail("unterminated string");
    ++i;
    return true;
  }
  bool val(JVal* v, int depth) {
    if (depth > 64) return fail("nesting too deep");
    ws();
    if (i >= t.size()) return fail("unexpected end");
    char c = t[i];
    if (c == '{') {
      v->kind = JVal::kObj;
      ++i;
      ws();
      if (i < t.size() && t[i] == '}') { ++i; return true; }
      for (;;) {
        ws();
        std::string k;
        if (!str(&k)) return false;
        ws();
        if (i >= t.size() || t[i] != ':') return fail("expected ':'");
        ++i;
        JVal x;
        if (!val(&x, depth + 1)) return false;
        v->obj.emplace_back(std::move(k), std::move(x));
        ws();
        if (i < t.size() && t[i] == ',') { ++i; continue; }
        if (i < t.size() && t[i] == '}') { ++i; return true; }
        return fail("expected ',' or '}'");
      }
    }
    if (c == '[') {
      v->kind = JVal::kArr;
      ++i;
      ws();
      if (i < t.size() && t[i] == ']') { ++i; return true; }
      for (;;) {
        JVal x;
        if (!val(&x, depth + 1)) return false;
        v->arr.push_back(std::move(x));
        ws();
        if (i < t.size() && t[i] == ',') { ++i; continue; }
        if (i < t.size() && t[i] == ']') { ++i; return true; }
        return fail("expected ',' or ']'");
      }
    }
    if (c == '"') {
      v->kind = JVal::kStr;
      return str(&v->str);
    }
    if (t.compare(i, 4, "true") == 0) { v->kind = JVal::kBool; v->b = true; i += 4; return true; }
    if (t.compare(i, 5, "false") == 0) { v->kind = JVal::kBool; i += 5; return true; }
    if (t.compare(i, 4, "null") == 0) { v->kind = JVal::kNull; i += 4; return true; }
    const char* s = t.c_str() + i;
    char* e = nullptr;
    double d = std::strtod(s, &e);
    if (e == s) return fail("unexpected character");
    v->kind = JVal::kNum;
    v->num = d;
    i += (size_t)(e - s);
    return true;
  }
};

bool as_int_list(const JVal* v, std::vector<int64_t>* out) {
  if (!v || v->kind != JVal::kArr) return false;
  out->clear();
  for (const auto& x : v->arr) {
    if (x.kind != JVal::kNum || x.num != std::floor(x.num)) return false;
    out->push_back((int64_t)x.num);
  }
  return true;
}

const char* kRatioFeatures[] = {"density", "run_coverage", "row_imbalance"};
const char* kIntFeatures[] = {"seq_q", "seq_kv", "batch_heads", "query_rows"};

bool known_feature(const std::string& n) {
  for (const char* f : kRatioFeatures)
    if (n == f) return true;
  for (const char* f : kIntFeatures)
    if (n == f) return true;
  return false;
}

bool read_ranking(const JVal* v, std::vector<int32_t>* rk, std::string* err) {
  std::vector<int64_t> ids;
  if (!as_int_list(v, &ids) || ids.empty()) { *err = "bad ranking"; return false; }
  rk->clear();
  for (int64_t id : ids) {
    if (!catalog_find((int32_t)id)) { *err = "ranking names an unknown plan"; return false; }
    rk->push_back((int32_t)id);
  }
  return true;
}

// Version 2: "features" lists the feature names; each regime has a "region",
// one [lo, hi] pair per feature with null for an unbounded side.
bool parse_regions(const JVal& root, Lut* out, std::string* err) {
  const JVal* feats = root.get("features");
  if (!feats || feats->kind != JVal::kArr || feats->arr.empty()) { *err = "missing feature list"; return false; }
  out->feature_names.clear();
  out->feature_edges.clear();
  for (const auto& f : feats->arr) {
    if (f.kind != JVal::kStr || !known_feature(f.str)) { *err = "unknown feature"; return false; }
    out->feature_names.push_back(f.str);
  }
  const size_t nf = out->feature_names.size();
  const JVal* regimes = root.get("regimes");
  if (!regimes || regimes->kind != JVal::kArr) { *err = "missing regimes"; return false; }
  out->regions.clear();
  for (const auto& r : regimes->arr) {
    std::vector<int64_t> key;
    const JVal* reg = r.kind == JVal::kObj ? r.get("region") : nullptr;
    if (r.kind != JVal::kObj || !as_int_list(r.get("key"), &key) || key.size() != 4 || !reg ||
        reg->kind != JVal::kArr || reg->arr.size() != nf) {
      *err = "bad regime entry";
      return false;
    }
    Lut::Region g;
    for (const auto& iv : reg->arr) {
      if (iv.kind != JVal::kArr || iv.arr.size() != 2) { *err = "bad region interval"; return false; }
      int64_t b[2] = {0, 0};
      char has[2] = {0, 0};
      for (int j = 0; j < 2; ++j) {
        const JVal& x = iv.arr[j];
        if (x.kind == JVal::kNull) continue;
        if (x.kind != JVal::kNum || x.num != std::floor(x.num)) { *err = "bad region bound"; return false; }
        b[j] = (int64_t)x.num;
        has[j] = 1;
      }
      if (has[0] && has[1] && b[1] <= b[0]) { *err = "empty region interval"; return false; }
      g.lo.push_back(b[0]);
      g.hi.push_back(b[1]);
      g.has_lo.push_back(has[0]);
      g.has_hi.push_back(has[1]);
    }
    if (!read_ranking(r.get("ranking"), &g.ranking, err)) return false;
    out->regions[key].push_back(std::move(g));
  }
  return true;
}

}  // namespace

bool lut_parse(const std::string& text, Lut* out, std::string* err) {
  JParser p(text);
  JVal root;
  if (!p.val(&root, 0)) { *err = "malformed JSON: " + p.err; return false; }
  p.ws();
  if (p.i != text.size()) { *err = "trailing characters after the artifact"; return false; }
  if (root.kind != JVal::kObj) { *err = "artifact is not a JSON object"; return false; }
  const JVal* fmt = root.get("format");
  if (!fmt || fmt->kind != JVal::kStr || fmt->str != "bsa-plan-table") { *err = "not a bsa-plan-table artifact"; return false; }
  const JVal* ver = root.get("version");
  if (!ver || ver->kind != JVal::kNum || ((int)ver->num != 1 && (int)ver->num != 2)) {
    *err = "unsupported artifact version";
    return false;
  }
  out->version = (int)ver->num;
  const JVal* arch = root.get("arch");
  if (!arch || arch->kind != JVal::kStr || arch->str != "gfx950") { *err = "artifact is not for gfx950"; return false; }
  out->arch = arch->str;
  // the catalog inside the artifact must match the library's catalog
  const JVal* cat = root.get("catalog");
  if (!cat || cat->kind != JVal::kArr || cat->arr.size() != catalog().size()) {
    *err = "artifact catalog does not match this library";
    return false;
  }
  for (size_t k = 0; k < cat->arr.size(); ++k) {
    std::vector<int64_t> e;
    if (!as_int_list(&cat->arr[k], &e) || e.size() != 7) { *err = "bad catalog entry"; return false; }
    const CatalogEntry& c = catalog()[k];
    if (e[0] != c.id || e[1] != c.tq || e[2] != c.tkv || e[3] != c.split || e[4] != c.stages || e[5] != c.waves ||
        e[6] != c.xcd_group) {
      *err = "artifact catalog entry " + std::to_string(k) + " does not match this library";
      return false;
    }
  }
  if (out->version == 2) return parse_regions(root, out, err);
  const JVal* schema = root.get("schema");
  if (!schema || schema->kind != JVal::kArr) { *err = "missing feature schema"; return false; }
  out->feature_names.clear();
  out->feature_edges.clear();
  for (const auto& f : schema->arr) {
    if (f.kind != JVal::kArr || f.arr.size() != 2 || f.arr[0].kind != JVal::kStr) { *err = "bad schema entry"; return false; }
    if (!known_feature(f.arr[0].str)) { *err = "unknown feature " + f.arr[0].str; return false; }
    std::vector<int64_t> edges;
    if (!as_int_list(&f.arr[1], &edges)) { *err = "bad bucket edges"; return false; }
    for (size_t k = 1; k < edges.size(); ++k)
      if (edges[k] <= edges[k - 1]) { *err = "bucket edges must increase"; return false; }
    out->feature_names.push_back(f.arr[0].str);
    out->feature_edges.push_back(edges);
  }
  const JVal* regimes = root.get("regimes");
  if (!regimes || regimes->kind != JVal::kArr) { *err = "missing regimes"; return false; }
  out->table.clear();
  for (const auto& r : regimes->arr) {
    std::vector<int64_t> key, bucket, ranking;
    if (r.kind != JVal::kObj || !as_int_list(r.get("key"), &key) || key.size() != 4 ||
        !as_int_list(r.get("bucket"), &bucket) || bucket.size() != out->feature_names.size() ||
        !as_int_list(r.get("ranking"), &ranking) || ranking.empty()) {
      *err = "bad regime entry";
      return false;
    }
    std::vector<int32_t> rk;
    for (int64_t id : ranking) {
      if (!catalog_find((int32_t)id)) { *err = "ranking names an unknown plan"; return false; }
      rk.push_back((int32_t)id);
    }
    out->table[key][bucket] = rk;
  }
  return true;
}

namespace {

// Integer feature `n` of z.  query_rows is the number of logical query-block
// rows, batch x heads x ceil(seq_q / B_Q).
int64_t int_feature(const std::string& n, const bsa_regime_query& z) {
  if (n == "seq_q") return z.seq_q;
  if (n == "seq_kv") return z.seq_kv;
  if (n == "query_rows") return z.bq > 0 ? z.batch_heads * ((z.seq_q + z.bq - 1) / z.bq) : 0;
  return z.batch_heads;
}

bool is_ratio(const std::string& n) { return n == "density" || n == "run_coverage" || n == "row_imbalance"; }

// Ratio feature `n` of z as (numerator, denominator); a zero denominator
// reads as 0.  row_imbalance = max_row_nnz * query_rows / nnz.
void ratio_feature(const std::string& n, const bsa_regime_query& z, __int128* num, __int128* den) {
  if (n == "density") {
    *num = z.nnz;
    *den = z.blocks;
  } else if (n == "run_coverage") {
    *num = z.run_blocks;
    *den = z.nnz;
  } else {
    *num = (__int128)z.max_row_nnz * int_feature("query_rows", z);
    *den = z.nnz;
  }
  if (*den <= 0) {
    *num = 0;
    *den = 1;
  }
}

}  // namespace

std::vector<int64_t> lut_bucket(const Lut& lut, const bsa_regime_query& z) {
  std::vector<int64_t> b;
  for (size_t f = 0; f < lut.feature_names.size(); ++f) {
    const std::string& n = lut.feature_names[f];
    const auto& edges = lut.feature_edges[f];
    int64_t idx = 0;
    if (is_ratio(n)) {
      __int128 num, den;
      ratio_feature(n, z, &num, &den);
      for (int64_t e : edges)
        if (num * 10000 >= (__int128)e * den) ++idx;
    } else {
      const int64_t v = int_feature(n, z);
      for (int64_t e : edges)
        if (v >= e) ++idx;
    }
    b.push_back(idx);
  }
  return b;
}

namespace {

// feature `n` of z >= edge (ratio features exactly, edges in units of 1e-4)
bool feature_ge(const std::string& n, const bsa_regime_query& z, int64_t edge) {
  if (is_ratio(n)) {
    __int128 num, den;
    ratio_feature(n, z, &num, &den);
    return num * 10000 >= (__int128)edge * den;
  }
  return int_feature(n, z) >= edge;
}

}  // namespace

std::vector<int32_t> lut_ranking(const Lut* lut, const bsa_regime_query& z, bool* hit) {
  *hit = false;
  if (lut && lut->version == 2) {
    const std::vector<int64_t> key{z.bq, z.bkv, z.dtype, z.head_dim};
    auto it = lut->regions.find(key);
    if (it != lut->regions.end()) {
      for (const Lut::Region& g : it->second) {
        bool in = true;
        for (size_t f = 0; f < lut->feature_names.size() && in; ++f) {
          const std::string& n = lut->feature_names[f];
          if (g.has_lo[f] && !feature_ge(n, z, g.lo[f])) in = false;
          if (in && g.has_hi[f] && feature_ge(n, z, g.hi[f])) in = false;
        }
        if (in) {
          *hit = true;
          return g.ranking;
        }
      }
    }
  } else if (lut) {
    const std::vector<int64_t> key{z.bq, z.bkv, z.dtype, z.head_dim};
    auto it = lut->table.find(key);
    if (it != lut->table.end()) {
      auto jt = it->second.find(lut_bucket(*lut, z));
      if (jt != it->second.end()) {
        *hit = true;
        return jt->second;
      }
    }
  }
  const int32_t base = base_plan(z.bq, z.bkv);
  if (base < 0) return {};
  return {base};
}

}  // namespace bsa
