// Planning kernels for gfx950: the shared mask state mu(M) (block-CSR and
// mask statistics, Section 5.2), the physical mapping of the selected plan
// (Section 4.2) and its task organisation (Section 4.3).
//
// Row-oriented kernels give one 64-lane wavefront to one row.  A row is read
// 64 columns per step with coalesced byte loads; ballot masks carry the
// activity of the step, so counting, run detection and compaction are scalar
// bit operations on one 64-bit word.
#include "bsa_internal.h"

namespace bsa {

namespace {

constexpr int kRowsPerBlock = 4;  // wavefronts (rows) per 256-thread workgroup

__device__ inline int find_bh(const int64_t* row_base, int nbh, int64_t r) {
  int lo = 0, hi = nbh;  // row_base[lo] <= r < row_base[hi]
  while (hi - lo > 1) {
    int mid = (lo + hi) >> 1;
    if (row_base[mid] <= r) lo = mid; else hi = mid;
  }
  return lo;
}

__device__ inline uint64_t lanes_below(int lane) { return (lane == 0) ? 0ull : ((~0ull) >> (64 - lane)); }

// Logical rows read as 32-bit words, for masks whose rows are 4-byte
// aligned: a step covers 256 columns, lane l holding columns 4l .. 4l+3 (byte
// j of its word is column 4l + j), and four ballots, one per byte position,
// carry the step's activity.  Counts, runs and the compacted columns are the
// same as those of the byte-wise walk.
constexpr int kWordSteps = 4;  // word steps whose loads go out together

template <bool kFill>
__device__ inline void mask_row_words(const MaskStateArgs& a, const uint8_t* row, int nkb, int64_t out_base, int lane,
                                      int64_t r) {
  const uint32_t* row32 = reinterpret_cast<const uint32_t*>(row);
  const int nw = nkb >> 2;
  int64_t nnz = 0, run = 0;
  uint64_t carry = 0;  // activity of the column just before the current step
  for (int w00 = 0; w00 < nw; w00 += 64 * kWordSteps) {
    // the loads of kWordSteps steps (clamped addresses, none behind a branch)
    uint32_t xs[kWordSteps];
#pragma unroll
    for (int s = 0; s < kWordSteps; ++s) xs[s] = row32[min(w00 + 64 * s + lane, nw - 1)];
    const uint32_t xn = kFill ? 0u : row32[min(w00 + 64 * kWordSteps, nw - 1)];
#pragma unroll
    for (int s = 0; s < kWordSteps; ++s) {
      const int w0 = w00 + 64 * s;
      if (w0 >= nw) break;
      const int wi = w0 + lane;
      const uint32_t word = wi < nw ? xs[s] : 0u;
      uint64_t bb[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) bb[j] = __ballot(((word >> (8 * j)) & 0xFFu) != 0);
      if (kFill) {
        const uint64_t below = lanes_below(lane);
        int64_t pos = out_base + nnz + __popcll(bb[0] & below) + __popcll(bb[1] & below) +
                      __popcll(bb[2] & below) + __popcll(bb[3] & below);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if ((bb[j] >> lane) & 1ull) a.col_idx[pos++] = 4 * wi + j;
        }
      } else {
        // the first column after this step: byte 0 of the next step's lane 0
        uint64_t next;
        if (s + 1 < kWordSteps) {
          next = (w0 + 64 < nw && (__shfl(xs[s + 1], 0, 64) & 0xFFu) != 0) ? 1ull : 0ull;
        } else {
          next = (w0 + 64 < nw && (xn & 0xFFu) != 0) ? 1ull : 0ull;
        }
        const uint64_t left[4] = {(bb[3] << 1) | carry, bb[0], bb[1], bb[2]};
        const uint64_t right[4] = {bb[1], bb[2], bb[3], (bb[0] >> 1) | (next << 63)};
#pragma unroll
        for (int j = 0; j < 4; ++j) run += __popcll(bb[j] & (left[j] | right[j]));
        carry = bb[3] >> 63;
      }
      nnz += __popcll(bb[0]) + __popcll(bb[1]) + __popcll(bb[2]) + __popcll(bb[3]);
    }
  }
  if (!kFill && lane == 0) {
    a.counts[r] = (int32_t)nnz;
    a.runs[r] = (int32_t)run;
  }
}

// Logical rows: count (with statistics) or fill the block-CSR columns.
template <bool kFill>
__global__ __launch_bounds__(256) void mask_rows_kernel(MaskStateArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  if (r >= a.R) return;
  const int bh = find_bh(a.row_base, a.nbh, r);
  const int b = bh / a.H, h = bh - b * a.H;
  const HeadDesc hd = a.heads[h];
  const int64_t qb = r - a.row_base[bh];
  const uint8_t* row = a.mask + b * a.stride_b + hd.mask_off + qb * (int64_t)hd.nkb;
  const int64_t out_base = kFill ? a.row_ptr[r] : 0;
  if (a.wide) {
    mask_row_words<kFill>(a, row, hd.nkb, out_base, lane, r);
    return;
  }
  int64_t nnz = 0, run = 0;
  uint64_t carry = 0;  // activity of the column just before the current step
  for (int c0 = 0; c0 < hd.nkb; c0 += 64) {
    const int c = c0 + lane;
    const bool act = (c < hd.nkb) && row[c] != 0;
    const uint64_t bits = __ballot(act);
    if (kFill) {
      if (act) a.col_idx[out_base + nnz + __popcll(bits & lanes_below(lane))] = c;
    } else {
      const uint64_t next = (c0 + 64 < hd.nkb && row[c0 + 64] != 0) ? 1ull : 0ull;
      const uint64_t left = (bits << 1) | carry;        // column c-1 active
      const uint64_t right = (bits >> 1) | (next << 63);  // column c+1 active
      run += __popcll(bits & (left | right));
      carry = bits >> 63;
    }
    nnz += __popcll(bits);
  }
  if (!kFill && lane == 0) {
    a.counts[r] = (int32_t)nnz;
    a.runs[r] = (int32_t)run;
  }
}

// Statistics of mu(M) from the per-row counts: one workgroup per row chunk
// (a chunk never crosses a (b, h) boundary), so only a handful of atomics
// per chunk reach the shared per-segment counters.
constexpr int kStatThreads = 256;

__global__ __launch_bounds__(kStatThreads) void row_stats_kernel(MaskStateArgs a) {
  const RowChunk ch = a.chunks[blockIdx.x];
  unsigned long long nnz = 0, run = 0, mx = 0;
  for (int64_t r = ch.begin + threadIdx.x; r < ch.end; r += kStatThreads) {
    const unsigned long long c = (unsigned long long)a.counts[r];
    nnz += c;
    run += (unsigned long long)a.runs[r];
    mx = c > mx ? c : mx;
  }
  for (int off = 32; off > 0; off >>= 1) {
    nnz += __shfl_xor(nnz, off, 64);
    run += __shfl_xor(run, off, 64);
    const unsigned long long o = __shfl_xor(mx, off, 64);
    mx = o > mx ? o : mx;
  }
  __shared__ unsigned long long part[3][kStatThreads / 64];
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    part[0][w] = nnz;
    part[1][w] = run;
    part[2][w] = mx;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int i = 1; i < kStatThreads / 64; ++i) {
      nnz += part[0][i];
      run += part[1][i];
      mx = part[2][i] > mx ? part[2][i] : mx;
    }
    SegStats* st = a.seg_stats + ch.seg;
    atomicAdd(&st->nnz, nnz);
    atomicAdd(&st->run_blocks, run);
    atomicMax(&st->max_row_nnz, mx);
    atomicAdd(a.bh_nnz + ch.bh, nnz);
  }
}

// ---------------------------------------------------------------------------
// Exclusive scan int32 -> int64 with the total in out[n]; three passes:
// per-block sums, a one-block scan of those sums, per-block rescans.
constexpr int kScanThreads = 256;
constexpr int kScanItems = 8;
constexpr int kScanTile = kScanThreads * kScanItems;

__device__ inline int64_t block_exclusive_scan(int64_t x, int64_t* total) {
  __shared__ int64_t wsum[kScanThreads / 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int64_t incl = x;
  for (int off = 1; off < 64; off <<= 1) {
    int64_t y = __shfl_up(incl, off, 64);
    if (lane >= off) incl += y;
  }
  if (lane == 63) wsum[w] = incl;
  __syncthreads();
  int64_t before = 0, all = 0;
  for (int i = 0; i < kScanThreads / 64; ++i) {
    if (i < w) before += wsum[i];
    all += wsum[i];
  }
  __syncthreads();
  *total = all;
  return before + incl - x;
}

__global__ __launch_bounds__(kScanThreads) void scan_block_sums(const int32_t* in, int64_t n, int64_t* sums) {
  const int64_t base = (int64_t)blockIdx.x * kScanTile + threadIdx.x * kScanItems;
  int64_t s = 0;
  for (int i = 0; i < kScanItems; ++i)
    if (base + i < n) s += in[base + i];
  int64_t total;
  (void)block_exclusive_scan(s, &total);
  if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

__global__ __launch_bounds__(kScanThreads) void scan_sums(int64_t* sums, int64_t nblocks) {
  int64_t carry = 0;
  for (int64_t base = 0; base < nblocks; base += kScanThreads) {
    const int64_t i = base + threadIdx.x;
    const int64_t x = i < nblocks ? sums[i] : 0;
    int64_t total;
    const int64_t ex = block_exclusive_scan(x, &total);
    if (i < nblocks) sums[i] = carry + ex;
    carry += total;
  }
}

__global__ __launch_bounds__(kScanThreads) void scan_apply(const int32_t* in, int64_t n, const int64_t* sums,
                                                           int64_t* out) {
  const int64_t base = (int64_t)blockIdx.x * kScanTile + threadIdx.x * kScanItems;
  int64_t v[kScanItems];
  int64_t s = 0;
  for (int i = 0; i < kScanItems; ++i) {
    v[i] = (base + i < n) ? in[base + i] : 0;
    s += v[i];
  }
  int64_t total;
  int64_t run = sums[blockIdx.x] + block_exclusive_scan(s, &total);
  for (int i = 0; i < kScanItems; ++i) {
    if (base + i < n) out[base + i] = run;
    run += v[i];
  }
  if (base < n && base + kScanItems >= n) out[n] = run;  // the thread holding the last element
}

__global__ void zero_i64(int64_t* out) {
  if (threadIdx.x == 0) out[0] = 0;
}

// ---------------------------------------------------------------------------
constexpr int kMapBatch = 16;

// Physical mapping of one geometry segment (Section 4.2): tile (pq, pk) is
// active iff one of its member logical blocks is; bit a*gkv + c records
// member (a, c) for Coarsened tiles.
template <bool kFill>
__global__ __launch_bounds__(256) void map_rows_kernel(MapArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t rp = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  if (rp >= a.Rp) return;
  const int64_t per_b = (int64_t)a.nsh * a.npq;
  const int b = (int)(rp / per_b);
  const int j = (int)((rp / a.npq) % a.nsh);
  const int pq = (int)(rp % a.npq);
  const int h = a.seg_heads[j];
  const HeadDesc hd = a.heads[h];
  const uint8_t* mh = a.mask + b * a.stride_b + hd.mask_off;
  int qb0, nqm;
  if (a.gq > 1 || a.rq == 1) {
    qb0 = pq * a.gq;
    nqm = min(a.gq, a.nqb - qb0);
  } else {
    qb0 = pq / a.rq;
    nqm = 1;
  }
  const int64_t out_base = kFill ? a.tile_ptr[rp] : 0;
  int64_t n = 0;
  if (a.gkv == 1 && a.wide) {
    // One member block along KV per tile (Direct, Refined, Coarsened along Q,
    // and Q-coarsened / KV-refined), word-aligned rows: lane l reads blocks
    // 4l .. 4l+3 of a step of 256 blocks from each of the tile's nqm query
    // rows; member bit a of block kb is row a's activity there.  Every block
    // with a member active contributes its tiles kb * rkv .. kb * rkv + rkv - 1
    // that exist (< npk), in ascending order, all with the block's bits.
    const uint8_t* base = mh + (int64_t)qb0 * a.nkb;
    const int nw = a.nkb >> 2;
    for (int w0 = 0; w0 < nw; w0 += 64) {
      const int wi = w0 + lane;
      const int wc = min(wi, nw - 1);
      uint64_t mem[4] = {0ull, 0ull, 0ull, 0ull};
      for (int a0 = 0; a0 < nqm; a0 += 4) {
        // four rows' loads in flight at once (clamped rows, then masked)
        uint32_t x[4];
#pragma unroll
        for (int k = 0; k < 4; ++k)
          x[k] = reinterpret_cast<const uint32_t*>(base + (int64_t)min(a0 + k, nqm - 1) * a.nkb)[wc];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint32_t word = (wi < nw && a0 + k < nqm) ? x[k] : 0u;
#pragma unroll
          for (int j = 0; j < 4; ++j)
            mem[j] |= (((word >> (8 * j)) & 0xFFu) != 0 ? 1ull : 0ull) << (a0 + k);
        }
      }
      uint64_t bb[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) bb[j] = __ballot(mem[j] != 0);
      // Every block has rkv tiles except perhaps the row's last one (byte 3
      // of word nw - 1), which has `deficit` fewer.  Tiles of the active
      // blocks of the lanes below come first, then this lane's in order.
      const uint64_t below = lanes_below(lane);
      const int deficit = a.rkv - (a.npk - (a.nkb - 1) * a.rkv);
      const int lw = nw - 1 - w0;  // lane holding the last block, if in this step
      const bool last_active = lw >= 0 && lw < 64 && ((bb[3] >> lw) & 1ull);
      int64_t before = (int64_t)a.rkv * (__popcll(bb[0] & below) + __popcll(bb[1] & below) +
                                         __popcll(bb[2] & below) + __popcll(bb[3] & below));
      if (last_active && lw < lane) before -= deficit;
      const int64_t pos = out_base + n + before;
      int64_t mine = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if ((bb[j] >> lane) & 1ull) {
          const int kb = 4 * wi + j;
          const int nt = min(a.rkv, a.npk - kb * a.rkv);
          if (kFill) {
            for (int s2 = 0; s2 < nt; ++s2) {
              a.tile_kv[pos + mine + s2] = kb * a.rkv + s2;
              if (a.member) a.member[pos + mine + s2] = mem[j];
            }
          }
          mine += nt;
        }
      }
      // this step's tile total
      n += (int64_t)a.rkv * (__popcll(bb[0]) + __popcll(bb[1]) + __popcll(bb[2]) + __popcll(bb[3])) -
           (last_active ? deficit : 0);
    }
    if (!kFill && lane == 0) a.counts[rp] = (int32_t)n;
    return;
  }
  if (a.gq == 1 && a.gkv == 1) {
    // Direct and Refined: one member per tile, the block (qb0, pk / rkv).
    // Every byte load of kMapBatch steps of 64 tiles is issued (from a
    // clamped address, so none sits behind a branch) before the first
    // ballot: a row costs one memory latency per 1024 tiles.
    const uint8_t* row = mh + (int64_t)qb0 * a.nkb;
    for (int p00 = 0; p00 < a.npk; p00 += 64 * kMapBatch) {
      uint8_t v[kMapBatch];
#pragma unroll
      for (int j = 0; j < kMapBatch; ++j) v[j] = row[min(p00 + 64 * j + lane, a.npk - 1) / a.rkv];
      bool act[kMapBatch];
#pragma unroll
      for (int j = 0; j < kMapBatch; ++j) act[j] = (p00 + 64 * j + lane < a.npk) && v[j] != 0;
#pragma unroll
      for (int j = 0; j < kMapBatch; ++j) {
        if (p00 + 64 * j >= a.npk) break;
        const uint64_t ball = __ballot(act[j]);
        if (kFill && act[j]) {
          const int64_t pos = out_base + n + __popcll(ball & lanes_below(lane));
          a.tile_kv[pos] = p00 + 64 * j + lane;
          if (a.member) a.member[pos] = 1ull;
        }
        n += __popcll(ball);
      }
    }
    if (!kFill && lane == 0) a.counts[rp] = (int32_t)n;
    return;
  }
  for (int p0 = 0; p0 < a.npk; p0 += 64) {
    const int pk = p0 + lane;
    uint64_t bits = 0;
    if (pk < a.npk) {
      int kb0, nkm;
      if (a.gkv > 1 || a.rkv == 1) {
        kb0 = pk * a.gkv;
        nkm = min(a.gkv, a.nkb - kb0);
      } else {
        kb0 = pk / a.rkv;
        nkm = 1;
      }
      for (int ai = 0; ai < nqm; ++ai) {
        const uint8_t* row = mh + (int64_t)(qb0 + ai) * a.nkb + kb0;
        for (int ci = 0; ci < nkm; ++ci)
          if (row[ci]) bits |= 1ull << (ai * a.gkv + ci);
      }
    }
    const bool act = bits != 0;
    const uint64_t ball = __ballot(act);
    if (kFill && act) {
      const int64_t pos = out_base + n + __popcll(ball & lanes_below(lane));
      a.tile_kv[pos] = pk;
      if (a.member) a.member[pos] = bits;
    }
    n += __popcll(ball);
  }
  if (!kFill && lane == 0) a.counts[rp] = (int32_t)n;
}

// ---------------------------------------------------------------------------
// Task organisation (Section 4.3): physical row rs of the segment is cut into
// `split` contiguous slices [floor(s*n/S), floor((s+1)*n/S)); empty slices
// are dropped; a row without active tiles keeps one empty task.
__device__ inline void task_row(const TaskArgs& a, int64_t rs, int* bh, int* pq, int64_t* lo, int64_t* hi) {
  const int64_t per_b = (int64_t)a.nsh * a.npq;
  const int b = (int)(rs / per_b);
  const int j = (int)((rs / a.npq) % a.nsh);
  *pq = (int)(rs % a.npq);
  *bh = b * a.H + a.seg_heads[j];
  const int64_t row = a.direct ? a.row_base[*bh] + *pq : rs;
  *lo = a.tile_ptr[row];
  *hi = a.tile_ptr[row + 1];
}

__global__ __launch_bounds__(256) void task_count_kernel(TaskArgs a) {
  const int64_t rs = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (rs >= a.Rp) return;
  int bh, pq;
  int64_t lo, hi;
  task_row(a, rs, &bh, &pq, &lo, &hi);
  const int64_t n = hi - lo;
  a.counts[rs] = (int32_t)(n == 0 ? 1 : (n < a.split ? n : a.split));
}

__global__ __launch_bounds__(256) void task_fill_kernel(TaskArgs a) {
  const int64_t rs = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (rs >= a.Rp) return;
  int bh, pq;
  int64_t lo, hi;
  task_row(a, rs, &bh, &pq, &lo, &hi);
  const int64_t n = hi - lo;
  int64_t out = a.task_ptr ? a.task_ptr[rs] : rs;
  if (n == 0 || a.split == 1) {
    Task t{bh, pq, (int32_t)lo, (int32_t)hi, 0, 1, 0, 0};
    a.tasks[out] = t;
    return;
  }
  const int nsplit = (int)(n < a.split ? n : a.split);
  int s_out = 0;
  for (int s = 0; s < a.split; ++s) {
    const int64_t b0 = lo + (s * n) / a.split, b1 = lo + ((s + 1) * n) / a.split;
    if (b1 == b0) continue;
    Task t{bh, pq, (int32_t)b0, (int32_t)b1, s_out, nsplit, 0, 0};
    a.tasks[out + s_out] = t;
    ++s_out;
  }
}

inline unsigned grid_for(int64_t rows, int per_block) { return (unsigned)((rows + per_block - 1) / per_block); }

}  // namespace

hipError_t launch_mask_count(const MaskStateArgs& a, hipStream_t s) {
  if (a.R == 0) return hipSuccess;
  hipLaunchKernelGGL(mask_rows_kernel<false>, dim3(grid_for(a.R, kRowsPerBlock)), dim3(256), 0, s, a);
  if (a.nchunks > 0) hipLaunchKernelGGL(row_stats_kernel, dim3((unsigned)a.nchunks), dim3(kStatThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_mask_fill(const MaskStateArgs& a, hipStream_t s) {
  if (a.R == 0) return hipSuccess;
  hipLaunchKernelGGL(mask_rows_kernel<true>, dim3(grid_for(a.R, kRowsPerBlock)), dim3(256), 0, s, a);
  return hipGetLastError();
}

int64_t scan_tmp_elems(int64_t n) { return (n + kScanTile - 1) / kScanTile + 1; }

hipError_t launch_scan_i32(const int32_t* in, int64_t* out, int64_t n, int64_t* block_tmp, hipStream_t s) {
  if (n == 0) {
    hipLaunchKernelGGL(zero_i64, dim3(1), dim3(64), 0, s, out);
    return hipGetLastError();
  }
  const int64_t nb = (n + kScanTile - 1) / kScanTile;
  hipLaunchKernelGGL(scan_block_sums, dim3((unsigned)nb), dim3(kScanThreads), 0, s, in, n, block_tmp);
  hipLaunchKernelGGL(scan_sums, dim3(1), dim3(kScanThreads), 0, s, block_tmp, nb);
  hipLaunchKernelGGL(scan_apply, dim3((unsigned)nb), dim3(kScanThreads), 0, s, in, n, block_tmp, out);
  return hipGetLastError();
}

hipError_t launch_map_count(const MapArgs& a, hipStream_t s) {
  if (a.Rp == 0) return hipSuccess;
  hipLaunchKernelGGL(map_rows_kernel<false>, dim3(grid_for(a.Rp, kRowsPerBlock)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_map_fill(const MapArgs& a, hipStream_t s) {
  if (a.Rp == 0) return hipSuccess;
  hipLaunchKernelGGL(map_rows_kernel<true>, dim3(grid_for(a.Rp, kRowsPerBlock)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_task_count(const TaskArgs& a, hipStream_t s) {
  if (a.Rp == 0) return hipSuccess;
  hipLaunchKernelGGL(task_count_kernel, dim3(grid_for(a.Rp, 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_task_fill(const TaskArgs& a, hipStream_t s) {
  if (a.Rp == 0) return hipSuccess;
  hipLaunchKernelGGL(task_fill_kernel, dim3(grid_for(a.Rp, 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace bsa
