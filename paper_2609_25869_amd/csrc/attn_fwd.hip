// Block-sparse attention forward for gfx950 (CDNA4): one workgroup per task,
// NWAVES wavefronts of 32 query rows each (T_Q = 32 * NWAVES), K/V tiles of
// TKV tokens streamed through a two-stage LDS ring (Sections 2.3, 4.2, 4.3).
//
// Layout of the work inside a wavefront
//   The score tile is computed transposed, S^T = K Q^T, with
//   v_mfma_f32_32x32x16_bf16 (A = K rows from LDS, B = the wave's Q rows held
//   in registers).  In the MFMA result each lane owns one query row
//   (lane % 32) and 16 keys per 32-key block, so the row max needs one
//   exchange between the two lane halves and the online-softmax state
//   (running max m, partial sum l) is per lane.  The output is accumulated
//   transposed as well, O^T += V^T P^T: the B operand is the lane's own
//   probabilities (no data movement, the key order inside an MFMA is chosen
//   to match the S^T layout) and the A operand is read from the row-major V
//   tile with ds_read_b64_tr_b16, which hands each lane 4 keys of one
//   head-dim column.  Rescaling O by exp2(m_old - m_new) is therefore a
//   per-lane multiply.
//
// LDS layout
//   K and V tiles arrive by direct global->LDS loads (no register staging)
//   and are stored row-major, 256 bytes (128 bf16) per token, with
//   the 16-byte chunks of row r permuted by chunk ^ f(r),
//   f(r) = swap of the two 2-bit halves of r % 16.  K operand reads (16
//   consecutive rows, one chunk) and V transposed reads (4 rows x 4 chunks
//   per 16-lane group) then touch distinct bank groups.
//
// Numerics: bf16 inputs, fp32 scores and softmax state, scores scaled by
// log2(e)/sqrt(d) so exp2 is used; P is rounded to bf16 for the PV product;
// O is normalised in fp32 and rounded to bf16 (RNE).  Masked entries
// (outside the tile's active members, or beyond the sequence end) are -inf
// before the max; a row whose running max is still -inf uses 0 as its
// reference so no NaN can arise (it keeps l = 0 and O = 0).
#include "bsa_internal.h"

namespace bsa {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kD = kHeadDim;
constexpr int kRowBytes = kD * 2;  // 256 bytes per token row in LDS
constexpr float kNegInf = -__builtin_huge_valf();

__device__ inline int swz(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }

__device__ inline f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ inline i16x4 lds_read_tr(const uint8_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p));
}

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// wait for this wave's outstanding vector-memory operations (the LDS DMA of
// the next tile); gfx9 s_waitcnt encoding with expcnt and lgkmcnt at maximum
__device__ inline void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

template <int NWAVES, int TKV>
struct Cfg {
  static constexpr int kThreads = 64 * NWAVES;
  static constexpr int kTQ = 32 * NWAVES;
  static constexpr int kNKB = TKV / 32;                 // 32-key blocks per tile
  static constexpr int kTileBytes = TKV * kRowBytes;
};

// Map the launch slot to a task so that each XCD (slot % 8) walks its own
// contiguous range of the task list.
__device__ inline int64_t task_of_slot(int64_t slot, int64_t nt) {
  const int64_t per = (nt + 7) / 8;
  const int64_t xcd = slot & 7, local = slot >> 3;
  if (local >= per) return -1;
  const int64_t t = xcd * per + local;
  return t < nt ? t : -1;
}

template <int NWAVES, int TKV>
__global__ __launch_bounds__(64 * NWAVES) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_fwd_kernel(AttnArgs a) {
  using C = Cfg<NWAVES, TKV>;
  // two pipeline stages, each a K tile and a V tile (separate arrays so the
  // compiler can tell the stage being filled from the stage being read)
  __shared__ __attribute__((aligned(1024))) uint8_t k0s[C::kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t v0s[C::kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t k1s[C::kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t v1s[C::kTileBytes];

  const int64_t nt = a.ntasks_dev ? *a.ntasks_dev : a.ntasks;
  const int64_t ti = task_of_slot(blockIdx.x, nt);
  if (ti < 0) return;
  const Task task = a.tasks[ti];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int n = lane & 31;   // query row of this lane inside the wave
  const int hh = lane >> 5;  // lane half
  const int b = task.bh / a.H, h = task.bh - b * a.H;
  const int q0 = task.pq * C::kTQ;
  const int qrow = q0 + 32 * w + n;

  // ---- Q fragment: B operand of S^T = K Q^T, lane (n, hh) holds d = 16c + 8hh .. +8
  bf16x8 qf[8];
  {
    const uint16_t* qp = a.q + b * a.qs0 + h * a.qs1 + (int64_t)qrow * a.qs2;
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      if (qrow < a.Nq) {
        qf[c] = *reinterpret_cast<const bf16x8*>(qp + 16 * c + 8 * hh);
      } else {
        qf[c] = bf16x8{};
      }
    }
  }

  const uint16_t* kbase = a.k + b * a.ks0 + h * a.ks1;
  const uint16_t* vbase = a.v + b * a.vs0 + h * a.vs1;

  // Direct global -> LDS loads: one instruction moves 64 lanes x 16 bytes =
  // 4 token rows into 1 KB of LDS, lane i landing at byte 16 * i.  Lane i of
  // load j therefore owns LDS row rr = 4 * (w + j * NWAVES) + i / 16 and
  // physical chunk i % 16, and fetches the logical chunk that the swizzle
  // places there.  Rows past the sequence end read a zero page.
  constexpr int kLoadsPerWave = TKV / (4 * NWAVES);
  static_assert(kLoadsPerWave >= 1 && TKV % (4 * NWAVES) == 0, "tile rows must split over the waves");
  int64_t src_off[kLoadsPerWave];  // element offset of this lane's chunk inside a token-row block
  int src_row[kLoadsPerWave];
#pragma unroll
  for (int j = 0; j < kLoadsPerWave; ++j) {
    const int rr = 4 * (w + j * NWAVES) + (lane >> 4);
    const int ch = (lane & 15) ^ swz(rr & 15);
    src_row[j] = rr;
    src_off[j] = ch * 8;
  }
  auto issue_tile = [&](int tile, uint8_t* kd, uint8_t* vd) {
    const int kv0 = a.kv_tile[tile] * TKV;
#pragma unroll
    for (int j = 0; j < kLoadsPerWave; ++j) {
      const int tok = kv0 + src_row[j];
      const bool ok = tok < a.Nkv;
      const uint16_t* kp = ok ? kbase + (int64_t)tok * a.ks2 + src_off[j] : a.zero_page;
      const uint16_t* vp = ok ? vbase + (int64_t)tok * a.vs2 + src_off[j] : a.zero_page;
      const int dst = 1024 * (w + j * NWAVES);
      __builtin_amdgcn_global_load_lds(kp, (__attribute__((address_space(3))) void*)(kd + dst), 16, 0, 0);
      __builtin_amdgcn_global_load_lds(vp, (__attribute__((address_space(3))) void*)(vd + dst), 16, 0, 0);
    }
  };

  // lane-constant LDS offsets
  const int sw = swz(lane & 15);
  int koff[8];  // K operand: row (lane % 32) of a 32-key block, chunk 2c + hh
#pragma unroll
  for (int c = 0; c < 8; ++c) koff[c] = (lane & 31) * kRowBytes + (((2 * c + hh) ^ sw) << 4);
  int voff[2][4];  // V transposed read: [r][dblk]
  {
    const int s16 = lane & 15, g = lane >> 4, mh = g & 1, gh = g >> 1;
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int row = 8 * r + 4 * gh + (s16 >> 2);  // within a 16-key chunk
#pragma unroll
      for (int dblk = 0; dblk < 4; ++dblk) {
        const int dcol = dblk * 32 + 16 * mh + 4 * (s16 & 3);
        voff[r][dblk] = row * kRowBytes + (((dcol >> 3) ^ swz(row)) << 4) + (dcol & 7) * 2;
      }
    }
  }

  // membership decode for this lane's query row
  const int q_local = 32 * w + n;
  const int mem_row = (a.gq > 1) ? (q_local >> a.bq_shift) : 0;
  const int mem_bits = a.gq * a.gkv;
  const uint64_t full = (mem_bits >= 64) ? ~0ull : ((1ull << mem_bits) - 1);

  f32x16 o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) o[i] = f32x16{};
  float m_run = kNegInf, l_run = 0.f;

  auto step = [&](const uint8_t* ks, const uint8_t* vs, int tile) {
    // ---- S^T = K Q^T
    f32x16 s[C::kNKB];
#pragma unroll
    for (int kb = 0; kb < C::kNKB; ++kb) s[kb] = f32x16{};
#pragma unroll
    for (int c = 0; c < 8; ++c) {
#pragma unroll
      for (int kb = 0; kb < C::kNKB; ++kb) {
        const bf16x8 ka = *reinterpret_cast<const bf16x8*>(ks + kb * 32 * kRowBytes + koff[c]);
        s[kb] = mfma32(ka, qf[c], s[kb]);
      }
    }

    // ---- mask (tile members / sequence tail), scale, row max
    const int kv0 = a.kv_tile[tile] * TKV;
    const uint64_t bits = a.member ? a.member[tile] : full;
    const bool tail = kv0 + TKV > a.Nkv;
    float mx = kNegInf;
    if (tail || bits != full) {
      const uint64_t rowbits = (bits >> (mem_row * a.gkv));
#pragma unroll
      for (int kb = 0; kb < C::kNKB; ++kb) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int j = kb * 32 + (i >> 2) * 8 + hh * 4 + (i & 3);
          const int c = (a.gkv > 1) ? (j >> a.bkv_shift) : 0;
          const bool ok = (kv0 + j < a.Nkv) && ((rowbits >> c) & 1ull);
          const float x = ok ? s[kb][i] * a.scale_log2 : kNegInf;
          s[kb][i] = x;
          mx = fmaxf(mx, x);
        }
      }
    } else {
#pragma unroll
      for (int kb = 0; kb < C::kNKB; ++kb) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float x = s[kb][i] * a.scale_log2;
          s[kb][i] = x;
          mx = fmaxf(mx, x);
        }
      }
    }
    mx = fmaxf(mx, __shfl_xor(mx, 32));

    // ---- online softmax update
    const float m_new = fmaxf(m_run, mx);
    const float m_use = (m_new == kNegInf) ? 0.f : m_new;
    const float alpha = fast_exp2(m_run - m_use);
    m_run = m_new;
    float rs = 0.f;
#pragma unroll
    for (int kb = 0; kb < C::kNKB; ++kb) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float p = fast_exp2(s[kb][i] - m_use);
        s[kb][i] = p;
        rs += p;
      }
    }
    l_run = l_run * alpha + rs;
#pragma unroll
    for (int d = 0; d < 4; ++d) o[d] *= alpha;

    // ---- O^T += V^T P^T
#pragma unroll
    for (int t = 0; t < TKV / 16; ++t) {
      bf16x8 pb;
#pragma unroll
      for (int e = 0; e < 8; ++e) pb[e] = (__bf16)s[t >> 1][8 * (t & 1) + e];
#pragma unroll
      for (int dblk = 0; dblk < 4; ++dblk) {
        const i16x4 lo = lds_read_tr(vs + t * 16 * kRowBytes + voff[0][dblk]);
        const i16x4 hi = lds_read_tr(vs + t * 16 * kRowBytes + voff[1][dblk]);
        const bf16x4 lo4 = __builtin_bit_cast(bf16x4, lo);
        const bf16x4 hi4 = __builtin_bit_cast(bf16x4, hi);
        bf16x8 va;
        va[0] = lo4[0]; va[1] = lo4[1]; va[2] = lo4[2]; va[3] = lo4[3];
        va[4] = hi4[0]; va[5] = hi4[1]; va[6] = hi4[2]; va[7] = hi4[3];
        o[dblk] = mfma32(va, pb, o[dblk]);
      }
    }
  };

  // two-stage ring: while one stage is consumed the next tile streams into
  // the other; one barrier per tile
  const int nkv_tiles = task.tile_end - task.tile_begin;
  if (nkv_tiles > 0) {
    issue_tile(task.tile_begin, k0s, v0s);
    wait_vmem();
    __syncthreads();
  }
  for (int it = 0; it < nkv_tiles; it += 2) {
    const int tile = task.tile_begin + it;
    if (it + 1 < nkv_tiles) issue_tile(tile + 1, k1s, v1s);
    step(k0s, v0s, tile);
    wait_vmem();
    __syncthreads();
    if (it + 1 >= nkv_tiles) break;
    if (it + 2 < nkv_tiles) issue_tile(tile + 2, k0s, v0s);
    step(k1s, v1s, tile + 1);
    wait_vmem();
    __syncthreads();
  }

  // ---- epilogue
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (task.nsplit == 1) {
    if (qrow < a.Nq) {
      const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
      uint16_t* op = a.o + b * a.os0 + h * a.os1 + (int64_t)qrow * a.os2;
#pragma unroll
      for (int dblk = 0; dblk < 4; ++dblk) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          bf16x4 v4;
#pragma unroll
          for (int e = 0; e < 4; ++e) v4[e] = (__bf16)(o[dblk][4 * g + e] * inv);
          *reinterpret_cast<bf16x4*>(op + dblk * 32 + 8 * g + 4 * hh) = v4;
        }
      }
      if (a.lse && hh == 0) {
        const float m_use = (m_run == kNegInf) ? 0.f : m_run;
        a.lse[((int64_t)b * a.H + h) * a.Nq + qrow] =
            l_tot > 0.f ? (m_use + __log2f(l_tot)) * 0.69314718055994530942f : kNegInf;
      }
    }
  } else {
    // Split-K partial state: m (log2 domain, raw), l, O unnormalised
    float* slot = a.ws + ti * (int64_t)C::kTQ * (kD + 2);
    if (hh == 0) {
      slot[q_local] = m_run;
      slot[C::kTQ + q_local] = l_tot;
    }
    float* os = slot + 2 * C::kTQ + (int64_t)q_local * kD;
#pragma unroll
    for (int dblk = 0; dblk < 4; ++dblk) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        f32x4 v4;
#pragma unroll
        for (int e = 0; e < 4; ++e) v4[e] = o[dblk][4 * g + e];
        *reinterpret_cast<f32x4*>(os + dblk * 32 + 8 * g + 4 * hh) = v4;
      }
    }
  }
}

// Split-K merge (Section 4.3, Fig. 5): rescale the partial states of one
// physical query row to their common maximum, sum, normalise, store bf16.
template <int TQ>
__global__ __launch_bounds__(256) void splitk_merge_kernel(AttnArgs a) {
  const int64_t nt = a.ntasks_dev ? *a.ntasks_dev : a.ntasks;
  const int64_t ti = blockIdx.x;
  if (ti >= nt) return;
  const Task task = a.tasks[ti];
  if (task.nsplit <= 1 || task.split != 0) return;
  const int b = task.bh / a.H, h = task.bh - b * a.H;
  const int64_t slot_elems = (int64_t)TQ * (kD + 2);
  const float* base = a.ws + ti * slot_elems;
  // 256 threads: each handles one query row and 32 head-dim columns per step
  for (int idx = threadIdx.x; idx < TQ * 4; idx += blockDim.x) {
    const int ql = idx >> 2, part = idx & 3;
    const int qrow = task.pq * TQ + ql;
    if (qrow >= a.Nq) continue;
    float mstar = kNegInf;
    for (int s = 0; s < task.nsplit; ++s) mstar = fmaxf(mstar, base[s * slot_elems + ql]);
    float acc[32];
#pragma unroll
    for (int e = 0; e < 32; ++e) acc[e] = 0.f;
    float L = 0.f;
    if (mstar != kNegInf) {
      for (int s = 0; s < task.nsplit; ++s) {
        const float* sl = base + s * slot_elems;
        const float ms = sl[ql];
        if (ms == kNegInf) continue;
        const float wgt = fast_exp2(ms - mstar);
        L += wgt * sl[TQ + ql];
        const float* os = sl + 2 * TQ + (int64_t)ql * kD + part * 32;
#pragma unroll
        for (int e = 0; e < 32; ++e) acc[e] += wgt * os[e];
      }
    }
    const float inv = L > 0.f ? 1.f / L : 0.f;
    uint16_t* op = a.o + b * a.os0 + h * a.os1 + (int64_t)qrow * a.os2 + part * 32;
#pragma unroll
    for (int e = 0; e < 32; e += 4) {
      bf16x4 v4;
#pragma unroll
      for (int u = 0; u < 4; ++u) v4[u] = (__bf16)(acc[e + u] * inv);
      *reinterpret_cast<bf16x4*>(op + e) = v4;
    }
    if (a.lse && part == 0)
      a.lse[((int64_t)b * a.H + h) * a.Nq + qrow] =
          L > 0.f ? (mstar + __log2f(L)) * 0.69314718055994530942f : kNegInf;
  }
}

template <int NWAVES, int TKV>
hipError_t launch_variant(const AttnArgs& a, hipStream_t s) {
  const int64_t slots = ((int64_t)a.ntasks + 7) / 8 * 8;
  if (slots == 0) return hipSuccess;
  hipLaunchKernelGGL((attn_fwd_kernel<NWAVES, TKV>), dim3((unsigned)slots), dim3(64 * NWAVES), 0, s, a);
  return hipGetLastError();
}

}  // namespace

bool attention_variant_exists(int tq, int tkv) {
  return (tq == 64 || tq == 128 || tq == 256) && (tkv == 32 || tkv == 64);
}

hipError_t launch_attention(int tq, int tkv, const AttnArgs& a, hipStream_t s) {
  if (tq == 64 && tkv == 32) return launch_variant<2, 32>(a, s);
  if (tq == 64 && tkv == 64) return launch_variant<2, 64>(a, s);
  if (tq == 128 && tkv == 32) return launch_variant<4, 32>(a, s);
  if (tq == 128 && tkv == 64) return launch_variant<4, 64>(a, s);
  if (tq == 256 && tkv == 32) return launch_variant<8, 32>(a, s);
  if (tq == 256 && tkv == 64) return launch_variant<8, 64>(a, s);
  return hipErrorInvalidValue;
}

hipError_t launch_splitk_merge(int tq, const AttnArgs& a, hipStream_t s) {
  if (a.ntasks == 0) return hipSuccess;
  const dim3 grid((unsigned)a.ntasks), block(256);
  if (tq == 64) hipLaunchKernelGGL(splitk_merge_kernel<64>, grid, block, 0, s, a);
  else if (tq == 128) hipLaunchKernelGGL(splitk_merge_kernel<128>, grid, block, 0, s, a);
  else if (tq == 256) hipLaunchKernelGGL(splitk_merge_kernel<256>, grid, block, 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace bsa
