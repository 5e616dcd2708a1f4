// Mean-pooled top-k block sparsifier on gfx950 (the step that supplies the
// logical mask M and its geometry B, Section 2.1), so that sparsify -> plan ->
// forward runs on the device.
//
// For every (b, h) and query block qb the score of KV block kb is the dot
// product of the mean query row of qb and the mean key row of kb; the k
// largest scores of each row are active (ties to the lower kb), and
// optionally every block the token diagonal passes through.  The selection
// is an integer decided by floating point, so the arithmetic is pinned:
// block sums of bf16 values in IEEE double (exact for these magnitudes), the
// mean as one double division, and each score accumulated over the head
// dimension in increasing order with one rounding per multiply and per add
// (contraction into fused multiply-adds is switched off).  Any
// implementation that follows the same steps selects the same blocks.
//
// Kernels (all HBM- or latency-bound; the attention kernel dominates):
//   block_mean_kernel    one workgroup per (b, h, block): 128 threads, one per
//                        head-dim column, sum the block's rows in order
//   block_score_kernel   64 x 64 score tiles, operand chunks staged in LDS,
//                        each thread 4 x 4 scores
//   topk_select_kernel   one workgroup per score row: MSB-first radix select
//                        of the k-th largest score (8 passes of 8 bits over
//                        order-preserving 64-bit keys held in LDS), ties ranked
//                        by column with a workgroup prefix count, coalesced
//                        write of the mask row with the diagonal added
#include "bsa_internal.h"

namespace bsa {

namespace {

__device__ inline double bf16_to_f64(uint16_t b) { return (double)__uint_as_float((uint32_t)b << 16); }

__global__ __launch_bounds__(128) void block_mean_kernel(const uint16_t* x, int64_t s0, int64_t s1, int64_t s2,
                                                         int32_t H, int32_t n, int32_t blk, int32_t nb, int32_t bh0,
                                                         double* out) {
  const int64_t w = blockIdx.x;  // (bh - bh0) * nb + i
  const int32_t i = (int32_t)(w % nb), bh = bh0 + (int32_t)(w / nb);
  const int32_t b = bh / H, h = bh - b * H;
  const int c = threadIdx.x;
  const uint16_t* p = x + b * s0 + h * s1 + c;
  const int32_t r0 = i * blk, r1 = min(n, r0 + blk);
  // rows in increasing order; eight loads go out before their additions
  double s = 0.0;
  int32_t r = r0;
  for (; r + 8 <= r1; r += 8) {
    double v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = bf16_to_f64(p[(int64_t)(r + j) * s2]);
#pragma unroll
    for (int j = 0; j < 8; ++j) s += v[j];
  }
  for (; r < r1; ++r) s += bf16_to_f64(p[(int64_t)r * s2]);
  out[w * kHeadDim + c] = s / (double)(r1 - r0);
}

constexpr int kST = 64;   // score tile edge
constexpr int kSC = 32;   // head-dim chunk staged per step

__global__ __launch_bounds__(256) void block_score_kernel(const double* pq, const double* pk, int32_t nqb,
                                                          int32_t nkb, double* scores) {
#pragma clang fp contract(off)
  __shared__ double sq[kST][kSC + 1];
  __shared__ double sk[kST][kSC + 1];
  const int64_t bhl = blockIdx.z;
  const int32_t q0 = blockIdx.y * kST, k0 = blockIdx.x * kST;
  const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
  double acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.0;
  }
  for (int c0 = 0; c0 < kHeadDim; c0 += kSC) {
    for (int idx = threadIdx.x; idx < kST * kSC; idx += 256) {
      const int r = idx / kSC, cc = idx % kSC;
      sq[r][cc] = (q0 + r < nqb) ? pq[(bhl * nqb + q0 + r) * kHeadDim + c0 + cc] : 0.0;
      sk[r][cc] = (k0 + r < nkb) ? pk[(bhl * nkb + k0 + r) * kHeadDim + c0 + cc] : 0.0;
    }
    __syncthreads();
    for (int cc = 0; cc < kSC; ++cc) {
      double a[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = sq[ty + 16 * i][cc];
#pragma unroll
      for (int j = 0; j < 4; ++j) bv[j] = sk[tx + 16 * j][cc];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const double prod = a[i] * bv[j];
          acc[i][j] = acc[i][j] + prod;
        }
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int32_t qb = q0 + ty + 16 * i;
    if (qb >= nqb) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int32_t kb = k0 + tx + 16 * j;
      if (kb < nkb) scores[(bhl * nqb + qb) * nkb + kb] = acc[i][j];
    }
  }
}

// Order-preserving map of a double to an unsigned key (larger score, larger
// key); -0 and +0 map to the same key, as they compare equal.
__device__ inline uint64_t order_key(double x) {
  if (x == 0.0) x = 0.0;
  const uint64_t u = (uint64_t)__double_as_longlong(x);
  return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

// Inclusive prefix sum over the 64 lanes of a wave.
__device__ inline uint32_t wave_inclusive_scan(uint32_t x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  return x;
}

__global__ __launch_bounds__(256) void topk_select_kernel(const double* scores, int32_t nqb, int32_t nkb, int32_t k,
                                                          int32_t diagonal, int32_t nq, int32_t nkv, int32_t bq,
                                                          int32_t bkv, int32_t bh0, uint8_t* mask) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  uint64_t* keys = reinterpret_cast<uint64_t*>(smem);
  uint8_t* take = smem + (size_t)nkb * 8;
  __shared__ uint32_t hist[256];
  __shared__ uint32_t chunk_ties[256];
  __shared__ uint64_t s_prefix;
  __shared__ int32_t s_remaining;
  const int tid = threadIdx.x;
  const int64_t row = blockIdx.x;  // (bh - bh0) * nqb + qb
  const int32_t qb = (int32_t)(row % nqb);
  const double* srow = scores + row * nkb;
  for (int32_t kb = tid; kb < nkb; kb += 256) keys[kb] = order_key(srow[kb]);
  __syncthreads();

  if (k >= nkb || k <= 0) {
    for (int32_t kb = tid; kb < nkb; kb += 256) take[kb] = k > 0;
  } else {
    // k-th largest key: fix one byte per pass from the most significant
    uint64_t prefix = 0, pmask = 0;
    int32_t remaining = k;  // rank of the sought key among those matching prefix
    for (int shift = 56; shift >= 0; shift -= 8) {
      hist[tid] = 0;
      __syncthreads();
      for (int32_t kb = tid; kb < nkb; kb += 256) {
        const uint64_t key = keys[kb];
        if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & 255], 1u);
      }
      __syncthreads();
      if (tid < 64) {
        // digit d of the sought key: the largest d whose keys, counted from
        // digit 255 down to d, reach `remaining` (d = 0 if none does before).
        // Lane l holds digits 255-4l .. 252-4l.
        uint32_t cnt[4], local = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          cnt[j] = hist[255 - 4 * tid - j];
          local += cnt[j];
        }
        const uint32_t incl = wave_inclusive_scan(local);
        const uint64_t reach = __ballot(incl >= (uint32_t)remaining || tid == 63);
        const int first = __builtin_ctzll(reach);
        if (tid == first) {
          int32_t above = (int32_t)(incl - local);
          int d = 255 - 4 * tid;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            if (d == 0 || above + (int32_t)cnt[j] >= remaining) break;
            above += (int32_t)cnt[j];
            --d;
          }
          s_remaining = remaining - above;
          s_prefix = prefix | ((uint64_t)d << shift);
        }
      }
      __syncthreads();
      remaining = s_remaining;
      prefix = s_prefix;
      pmask |= 0xFFull << shift;
    }
    // prefix is the k-th largest key; `remaining` of the keys equal to it are
    // taken, the lowest columns first
    const int32_t per = (nkb + 255) / 256;
    const int32_t c0 = min(nkb, tid * per), c1 = min(nkb, c0 + per);
    uint32_t ties = 0;
    for (int32_t kb = c0; kb < c1; ++kb) ties += keys[kb] == prefix;
    chunk_ties[tid] = ties;
    __syncthreads();
    if (tid < 64) {
      // exclusive prefix over the 256 chunks, four per lane
      uint32_t t[4], local = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        t[j] = chunk_ties[4 * tid + j];
        local += t[j];
      }
      uint32_t run = wave_inclusive_scan(local) - local;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        chunk_ties[4 * tid + j] = run;
        run += t[j];
      }
    }
    __syncthreads();
    int32_t rank = (int32_t)chunk_ties[tid];
    for (int32_t kb = c0; kb < c1; ++kb) {
      const uint64_t key = keys[kb];
      if (key == prefix) {
        take[kb] = rank < remaining;
        ++rank;
      } else {
        take[kb] = key > prefix;
      }
    }
  }
  __syncthreads();
  // the diagonal: columns [lo / bkv, (hi - 1) / bkv] for the row's tokens
  // [lo, hi) that also exist as keys
  const int32_t lo = qb * bq, hi = min(min(nq, nkv), lo + bq);
  const int32_t d0 = (diagonal && lo < hi) ? lo / bkv : 1, d1 = (diagonal && lo < hi) ? (hi - 1) / bkv : 0;
  uint8_t* out = mask + ((int64_t)bh0 * nqb + row) * nkb;
  for (int32_t kb = tid; kb < nkb; kb += 256) out[kb] = (take[kb] || (kb >= d0 && kb <= d1)) ? 1 : 0;
}

}  // namespace

// KV blocks per score row: the keys and flags of a row (9 bytes per block)
// stay within 64 KB of LDS
int32_t sparsify_max_kv_blocks() { return 6144; }

hipError_t launch_block_mean(const uint16_t* x, int64_t s0, int64_t s1, int64_t s2, int32_t H, int32_t n,
                             int32_t blk, int32_t bh0, int32_t nbh, double* out, hipStream_t s) {
  const int32_t nb = (n + blk - 1) / blk;
  const int64_t grid = (int64_t)nbh * nb;
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL(block_mean_kernel, dim3((unsigned)grid), dim3(128), 0, s, x, s0, s1, s2, H, n, blk, nb, bh0,
                     out);
  return hipGetLastError();
}

hipError_t launch_block_scores(const double* pq, const double* pk, int32_t nqb, int32_t nkb, int32_t nbh,
                               double* scores, hipStream_t s) {
  const dim3 grid((unsigned)((nkb + kST - 1) / kST), (unsigned)((nqb + kST - 1) / kST), (unsigned)nbh);
  hipLaunchKernelGGL(block_score_kernel, grid, dim3(256), 0, s, pq, pk, nqb, nkb, scores);
  return hipGetLastError();
}

hipError_t launch_topk_select(const double* scores, int32_t nqb, int32_t nkb, int32_t k, int32_t diagonal,
                              int32_t nq, int32_t nkv, int32_t bq, int32_t bkv, int32_t bh0, int32_t nbh,
                              uint8_t* mask, hipStream_t s) {
  const int64_t rows = (int64_t)nbh * nqb;
  if (rows == 0) return hipSuccess;
  const size_t lds = (size_t)nkb * 9;
  hipLaunchKernelGGL(topk_select_kernel, dim3((unsigned)rows), dim3(256), lds, s, scores, nqb, nkb, k, diagonal, nq,
                     nkv, bq, bkv, bh0, mask);
  return hipGetLastError();
}

}  // namespace bsa
