// Native catalog, eligibility and profile-guided regime selection (host).
#pragma once

#include <cstdint>
#include <map>
#include <string>
#include <vector>

#include "../../include/bsa.h"

namespace bsa {

// Catalog of gfx950 plans (Section 4.4): a physical tile (the mapping of
// Section 4.2) and an organization (Section 4.3): Split-K partitions, the
// kernel's wavefronts and ring depth, and the traversal order of the tasks
// over the eight XCDs (xcd_group XCDs share one stretch of the task list).
struct CatalogEntry {
  int32_t id, tq, tkv, split, stages, waves, xcd_group;
};

const std::vector<CatalogEntry>& catalog();
const CatalogEntry* catalog_find(int32_t id);

// Why a plan is not eligible, or nullptr when it is (Section 4.4).
const char* ineligible_reason(const CatalogEntry& e, int32_t bq, int32_t bkv, const bsa_shapes& s);

// Mapping kind of tile (tq, tkv) over block (bq, bkv): 0 Direct, 1 Coarsened,
// 2 Refined, 3 mixed.
int mapping_kind(int32_t bq, int32_t bkv, int32_t tq, int32_t tkv);

// Base plan of request key (bq, bkv): the split-free plan whose tile is
// nearest to the logical block (Direct when available), smallest id on ties.
// -1 if no catalog tile nests with the geometry.
int32_t base_plan(int32_t bq, int32_t bkv);

// Loaded plan-table artifact (Section 5.1).
struct Lut {
  int version = 0;
  std::string arch;
  // feature schema: names and bucket edges (ratio features in units of 1e-4)
  std::vector<std::string> feature_names;
  std::vector<std::vector<int64_t>> feature_edges;
  // version 1: (bq, bkv, dtype, head_dim) -> bucket tuple -> ranking
  std::map<std::vector<int64_t>, std::map<std::vector<int64_t>, std::vector<int32_t>>> table;
  // version 2: the regimes of a key are disjoint regions, one half-open
  // interval [lo, hi) per feature (has_lo / has_hi false = unbounded), the
  // leaves of a decision tree learned offline
  struct Region {
    std::vector<int64_t> lo, hi;
    std::vector<char> has_lo, has_hi;
    std::vector<int32_t> ranking;
  };
  std::map<std::vector<int64_t>, std::vector<Region>> regions;
};

// Parse an artifact; on failure returns false and fills *err.
bool lut_parse(const std::string& text, Lut* out, std::string* err);

// Bucket tuple of a regime query under the table's schema.
std::vector<int64_t> lut_bucket(const Lut& lut, const bsa_regime_query& z);

// Ranking for z: the regime's list on a hit, the base plan alone on a miss
// (Algorithm 2).  *hit reports which.
std::vector<int32_t> lut_ranking(const Lut* lut, const bsa_regime_query& z, bool* hit);

}  // namespace bsa
