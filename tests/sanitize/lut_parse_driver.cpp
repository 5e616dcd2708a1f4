// Host driver for the plan-table reader under AddressSanitizer and
// UndefinedBehaviorSanitizer: parses every file named on the command line
// (valid artifacts and damaged copies), and for each accepted table runs the
// regime lookup on a grid of queries.  Prints one line per file; exits 0
// unless a sanitizer stops it.
#include <cstdio>
#include <fstream>
#include <sstream>
#include <string>

#include "catalog.h"

int main(int argc, char** argv) {
  for (int i = 1; i < argc; ++i) {
    std::ifstream f(argv[i], std::ios::binary);
    std::ostringstream ss;
    ss << f.rdbuf();
    bsa::Lut lut;
    std::string err;
    const bool ok = bsa::lut_parse(ss.str(), &lut, &err);
    long lookups = 0, hits = 0;
    if (ok) {
      const int geoms[][2] = {{64, 64}, {128, 128}, {64, 32}, {32, 32}, {16, 16}, {128, 32}, {32, 128}, {256, 64}};
      for (const auto& g : geoms)
        for (long seq : {1L, 2048L, 65536L, 115200L, 1L << 30})
          for (long bh : {1L, 4L, 24L, 1000L})
            for (long nnz : {0L, 1L, 37L, 5000L, 1000000L}) {
              bsa_regime_query z{};
              z.bq = g[0];
              z.bkv = g[1];
              z.dtype = BSA_DTYPE_BF16;
              z.head_dim = 128;
              z.batch_heads = bh;
              z.seq_q = z.seq_kv = seq;
              z.nnz = nnz;
              z.blocks = nnz * 3 + (nnz == 0 ? 0 : 1);
              z.run_blocks = nnz / 2;
              bool hit = false;
              const auto r = bsa::lut_ranking(&lut, z, &hit);
              lookups += 1;
              hits += hit ? 1 : 0;
              if (r.empty() && bsa::base_plan(z.bq, z.bkv) >= 0) {
                std::printf("%s: empty ranking\n", argv[i]);
                return 2;
              }
            }
    }
    std::printf("%s: %s%s (%ld lookups, %ld hits)\n", argv[i], ok ? "accepted" : "rejected: ", ok ? "" : err.c_str(),
                lookups, hits);
  }
  return 0;
}
