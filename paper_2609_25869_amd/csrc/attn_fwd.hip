// Block-sparse attention forward for gfx950 (CDNA4): one workgroup per task,
// NWAVES wavefronts, each owning G groups of 32 query rows
// (T_Q = 32 * G * NWAVES), K/V tiles of TKV tokens streamed through LDS rings
// of STAGES slots (pipeline depth, Sections 2.3, 4.2, 4.3).  The loop is
// software pipelined: the scores of tile t+1 (MFMA) are computed while the
// probabilities of tile t (VALU) are formed and O accumulates P V of tile
// t-1, whose probabilities were checked at the end of the previous
// iteration.
//
// Layout of the work inside a wavefront
//   The score tile is computed transposed, S^T = K Q^T, with
//   v_mfma_f32_32x32x16_bf16 (A = K rows from LDS, B = a 32-row group of the
//   wave's Q rows held in registers).  In the MFMA result each lane owns one
//   query row (lane % 32) of the group and 16 keys per 32-key block, so the
//   row max needs one exchange between the two lane halves and the
//   online-softmax state (running max m, partial sum l) is per lane and
//   group.  The output is accumulated transposed as well, O^T += V^T P^T: the
//   B operand is the lane's own probabilities (no data movement, the key
//   order inside an MFMA is chosen to match the S^T layout) and the A operand
//   is read from the row-major V tile with ds_read_b64_tr_b16, which hands
//   each lane 4 keys of one head-dim column.  Rescaling O by
//   exp2(m_old - m_new) is therefore a per-lane multiply.
//   Every A operand read from LDS feeds G MFMAs, one per row group: with
//   G = 2 a wave holds 64 query rows, which halves the LDS reads and the K/V
//   traffic per flop (the register file then holds one wave per SIMD).
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
// log2(e)/sqrt(d) in fp32 so exp2 is used.  The running reference m of a
// row is not tracked tile by tile: the probabilities of a tile are formed
// against the current reference and their sum is checked before any MFMA
// consumes them; only when a probability may exceed 2^8 (or the row has
// no reference yet) is the tile's row maximum formed, the row's reference
// raised and its O rescaled.  That decision is taken per query row, from the
// row's own active scores.  P is rounded to bf16 for the PV product; O is
// normalised in fp32 and rounded to bf16 (RNE).  Masked entries (outside
// the tile's active members, or beyond the sequence end) are -inf before
// any of this; a row whose reference is still unset uses 0 as its
// reference, so no NaN can arise (it keeps l = 0 and O = 0).
#include "bsa_internal.h"
#include "slot_map.h"

namespace bsa {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kD = kHeadDim;
constexpr int kRowBytes = kD * 2;  // 256 bytes per token row in LDS
constexpr float kNegInf = -__builtin_huge_valf();

__device__ inline int swz(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }

__device__ inline f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// The same MFMA with the accumulator pinned to VGPRs and B read from AGPRs.
// Once a kernel needs more than 256 registers the compiler selects the AGPR
// form for every MFMA; score tiles are VALU operands, and from AGPRs each
// element would first need a copy.  The hardware does not interlock an MFMA
// result read by a VALU instruction, nor a VALU-written operand read by an
// MFMA, and the compiler inserts no wait states around inline assembly, so
// the callers keep those distances: the next MFMA of the same chain issues
// at least one other MFMA later, VALU reads of the scores follow a whole
// pipeline iteration later, and the two places where that does not hold by
// construction (the Q operands just written, the first tile's scores just
// computed) get an explicit wait (hazard_wait).
__device__ inline void mfma32_vacc(f32x16& acc, bf16x8 a, bf16x8 b, bool zero) {
  if (zero) {
    asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=&v"(acc) : "v"(a), "a"(b));
  } else {
    asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(acc) : "v"(a), "a"(b));
  }
}

// 24 wait states, tied to the registers they protect (the compiler can then
// move no producer after it and no consumer before it): more than an 8-pass
// MFMA result needs before a VALU read, and than a VALU write needs before an
// MFMA reads it.
template <typename T>
__device__ inline void hazard_wait_v(T& x) { asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" : "+v"(x)); }
// the same for the Q operands of a 64-row wave, all in one wait
__device__ inline void hazard_wait_q2(bf16x8 (&q)[2][8]) {
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7"
               : "+a"(q[0][0]), "+a"(q[0][1]), "+a"(q[0][2]), "+a"(q[0][3]), "+a"(q[0][4]), "+a"(q[0][5]),
                 "+a"(q[0][6]), "+a"(q[0][7]), "+a"(q[1][0]), "+a"(q[1][1]), "+a"(q[1][2]), "+a"(q[1][3]),
                 "+a"(q[1][4]), "+a"(q[1][5]), "+a"(q[1][6]), "+a"(q[1][7]));
}

__device__ inline i16x4 lds_read_tr(const uint8_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p));
}

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

template <int NWAVES, int G, int TKV>
struct Cfg {
  static constexpr int kThreads = 64 * NWAVES;
  static constexpr int kRowsPerWave = 32 * G;
  static constexpr int kTQ = kRowsPerWave * NWAVES;
  static constexpr int kNKB = TKV / 32;                 // 32-key blocks per tile
  static constexpr int kTileBytes = TKV * kRowBytes;
};

// Value of the same register in lane l ^ 32 (the other half of the wave).
__device__ inline uint32_t other_half_u32(uint32_t x) {
  const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  // lanes 0-31 find the partner in r[1], lanes 32-63 in r[0]; the other entry is x itself
  return (threadIdx.x & 32) ? r[0] : r[1];
}
__device__ inline float other_half(float x) { return __uint_as_float(other_half_u32(__float_as_uint(x))); }

// In-place updates for the rare paths (rescale, masking).  The tied
// operands pin each result to the register it came from; written as plain
// C++ the compiler gives the updated values new registers and then copies
// the whole accumulator on the common path where the update did not run.
// With G = 2 the accumulators live in AGPRs, which VALU instructions cannot
// address, and the multiply is left to the compiler.
template <bool kInVgpr>
__device__ inline void scale_inplace(f32x16& v, float alpha) {
  if constexpr (kInVgpr) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      float x = v[i];
      asm volatile("v_mul_f32_e32 %0, %1, %0" : "+v"(x) : "v"(alpha));
      v[i] = x;
    }
  } else {
    v *= alpha;
  }
}

// x = keep ? x : -inf, in place (keep is per lane)
__device__ inline void mask_inplace(float& x, bool keep) {
  const float ninf = -__builtin_huge_valf();
  asm volatile("v_cndmask_b32_e64 %0, %1, %0, %2" : "+v"(x) : "v"(ninf), "s"(__ballot(keep)));
}

// A row's reference is raised only when the probabilities of a tile, formed
// against it, sum to more than 2^8 in one lane; below that every
// probability is at most 2^8, which fp32 sums and bf16 P hold exactly as
// well, and the rescale of O is skipped.
constexpr float kSumMax = 256.0f;

// Wait until at most N of this wave's vector-memory operations (the LDS DMA
// of younger tiles) are outstanding and all of its LDS reads have retired
// (gfx9 s_waitcnt encoding: vmcnt in bits 3:0 and 15:14, expcnt 6:4 at its
// maximum, lgkmcnt 11:8 = 0).
template <int N>
__device__ inline void wait_vm_lgkm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt(0x0070 | (N & 15) | ((N >> 4) << 14));
}

// Workgroup barrier without a memory fence: LDS writes made by the DMA are
// complete once vmcnt says so, and a fence here would also drain the
// prefetches that are meant to stay in flight.  The empty asm statements
// keep the compiler from moving memory accesses across the barrier.
__device__ inline void block_sync() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Waves per SIMD the register budget is sized for: two for G = 1 with four
// or more waves per workgroup, and for 2-wave workgroups whose ring takes
// at most 32 KB (four of them share a CU); one for G = 2 (its accumulators
// and Q fragments need the whole register file) and for the 2-wave T_Q = 64
// workgroups with 64 KB rings, of which only two share a CU.
template <int NWAVES, int G, int TKV, int STAGES>
constexpr int waves_per_simd() { return (G == 1 && (NWAVES > 2 || TKV * STAGES <= 64)) ? 2 : 1; }

template <int NWAVES, int G, int TKV, int STAGES>
__global__ __launch_bounds__(64 * NWAVES)
__attribute__((amdgpu_waves_per_eu(waves_per_simd<NWAVES, G, TKV, STAGES>(), waves_per_simd<NWAVES, G, TKV, STAGES>())))
void attn_fwd_kernel(AttnArgs a) {
  using C = Cfg<NWAVES, G, TKV>;
  constexpr int kNKB = C::kNKB;
  static_assert(STAGES == 2 || STAGES == 4 || STAGES == 8, "ring depth");
  static_assert(G == 1 || G == 2, "row groups per wave");
  // A ring of STAGES slots; slot j holds K of a tile x = j (mod STAGES) and
  // V of tile x-2.  Iteration t reads slot (t+1) % STAGES: K of tile t+1
  // (scores of the next tile) and V of tile t-1 (O += P V of the previous
  // tile), and refills slot t % STAGES (read by iteration t-1) with K of
  // tile t+STAGES and V of tile t+STAGES-2, so every load has STAGES-2 whole
  // iterations plus the current one to arrive.  Each slot is its own array: the compiler then
  // sees that reads of one slot never alias the DMA filling another and
  // keeps those loads in flight.
  constexpr int kSlotBytes = 2 * C::kTileBytes;
  constexpr int kBytes4 = STAGES > 2 ? kSlotBytes : 16;   // slots 2-3
  constexpr int kBytes8 = STAGES > 4 ? kSlotBytes : 16;   // slots 4-7
  __shared__ __attribute__((aligned(1024))) uint8_t ring0[kSlotBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t ring1[kSlotBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t ring2[kBytes4];
  __shared__ __attribute__((aligned(1024))) uint8_t ring3[kBytes4];
  __shared__ __attribute__((aligned(1024))) uint8_t ring4[kBytes8];
  __shared__ __attribute__((aligned(1024))) uint8_t ring5[kBytes8];
  __shared__ __attribute__((aligned(1024))) uint8_t ring6[kBytes8];
  __shared__ __attribute__((aligned(1024))) uint8_t ring7[kBytes8];
  auto kslot = [&](int i) -> uint8_t* {
    switch (i) {
      case 0: return ring0;
      case 1: return ring1;
      case 2: return ring2;
      case 3: return ring3;
      case 4: return ring4;
      case 5: return ring5;
      case 6: return ring6;
      default: return ring7;
    }
  };
  auto vslot = [&](int i) -> uint8_t* { return kslot(i) + C::kTileBytes; };

  const int64_t nt = a.ntasks_dev ? *a.ntasks_dev : a.ntasks;
  int64_t ti = task_of_slot(blockIdx.x, nt, a.slot_group, a.slot_run, a.balanced ? a.share_lo : nullptr);
  if (ti < 0) return;
  if (a.order) ti = ((const __attribute__((address_space(4))) int32_t*)a.order)[ti];
  const Task task = a.tasks[ti];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index (uniform)
  const int n = lane & 31;   // query row of this lane inside a 32-row group
  const int hh = lane >> 5;  // lane half
  const int b = task.bh / a.H, h = task.bh - b * a.H;
  const int q0 = task.pq * C::kTQ;
  // row of group g inside the task's query tile, and in the sequence
  auto q_local = [&](int g) { return C::kRowsPerWave * w + 32 * g + n; };
  auto q_row = [&](int g) { return q0 + q_local(g); };

  // ---- Q fragments: B operands of S^T = K Q^T, lane (n, hh) of group g
  // holds d = 16c + 8hh .. +8 of its row
  const float c_log2 = a.scale_log2;
  bf16x8 qf[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int qr = q_row(g);
    const uint16_t* qp = a.q + b * a.qs0 + h * a.qs1 + (int64_t)(qr < a.Nq ? qr : 0) * a.qs2;
#pragma unroll
    for (int c = 0; c < 8; ++c) qf[g][c] = *reinterpret_cast<const bf16x8*>(qp + 16 * c + 8 * hh);
    if (qr >= a.Nq) {
#pragma unroll
      for (int c = 0; c < 8; ++c) qf[g][c] = bf16x8{};
    }
  }

  // The task's tile list and membership bits are read through the scalar
  // cache (constant address space): vector loads would be counted together
  // with the in-flight K/V loads and force them to drain.
  typedef const __attribute__((address_space(4))) int32_t* ci32p;
  typedef const __attribute__((address_space(4))) uint64_t* cu64p;
  const int tb = task.tile_begin;
  const int nkv_tiles = task.tile_end - tb;
  ci32p kvt = (ci32p)(a.kv_tile + tb);

  // ---- K/V tiles: buffer loads straight into LDS
  // One instruction moves 64 lanes x 16 bytes = 4 token rows into 1 KB of
  // LDS, lane i landing at byte 16 * i.  Lane i of load j owns LDS row
  // rr = 4 * (w + j * NWAVES) + i / 16 and physical chunk i % 16, and reads
  // the logical chunk that the swizzle places there.  One buffer descriptor
  // per tensor covers the head's Nkv tokens, so rows past the sequence end
  // read as zero with no extra instruction; a load's per-lane byte offset is
  // the lane's offset inside its row group plus the group's first token times
  // the token stride, in 32 bits (plan eligibility keeps one head's K/V rows
  // within 4 GiB).
  constexpr int kLoadsPerWave = TKV / (4 * NWAVES);
  static_assert(kLoadsPerWave >= 1 && TKV % (4 * NWAVES) == 0, "tile rows must split over the waves");
  const char* kbase = reinterpret_cast<const char*>(a.k + b * a.ks0 + h * a.ks1);
  const char* vbase = reinterpret_cast<const char*>(a.v + b * a.vs0 + h * a.vs1);
  const int64_t kstride = a.ks2 * 2, vstride = a.vs2 * 2;  // bytes per token
  // The swizzle depends on the row modulo 16, which repeats every kRep loads
  // of a wave; later loads reuse those lane offsets and add whole rows
  // through the scalar offset (which the descriptor's range check includes).
  constexpr int kRep = NWAVES % 4 == 0 ? 1 : 4 / (NWAVES % 4 == 2 ? 2 : 1);
  constexpr int kRepN = kRep < kLoadsPerWave ? kRep : kLoadsPerWave;
  uint32_t koffs[kRepN], voffs[kRepN];
#pragma unroll
  for (int j = 0; j < kRepN; ++j) {
    const int rr = 4 * (w + j * NWAVES) + (lane >> 4);
    const int ch = (lane & 15) ^ swz(rr & 15);
    koffs[j] = (uint32_t)(rr * kstride) + ch * 16;
    voffs[j] = (uint32_t)(rr * vstride) + ch * 16;
  }
  const __amdgpu_buffer_rsrc_t krsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(kbase), 0, (int)((int64_t)a.Nkv * kstride), 0x00020000);
  const __amdgpu_buffer_rsrc_t vrsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(vbase), 0, (int)((int64_t)a.Nkv * vstride), 0x00020000);
  // load j of this wave's share of the tile starting at token kv0
  auto dma_one = [&](__amdgpu_buffer_rsrc_t rsrc, int64_t stride, const uint32_t* offs, int kv0, int j,
                     uint8_t* dst_arr) {
    const uint32_t row0 = (uint32_t)(kv0 + (j / kRep) * (kRep * 4 * NWAVES)) * (uint32_t)stride;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rsrc, (__attribute__((address_space(3))) void*)(dst_arr + 1024 * (w + j * NWAVES)), 16, offs[j % kRep] + row0,
        0, 0, 0);
  };
  // copy the TKV tokens starting at kv0 into one ring slot
  auto dma_k = [&](int kv0, int slot) {
#pragma unroll
    for (int j = 0; j < kLoadsPerWave; ++j) dma_one(krsrc, kstride, koffs, kv0, j, kslot(slot));
  };
  auto dma_v = [&](int kv0, int slot) {
#pragma unroll
    for (int j = 0; j < kLoadsPerWave; ++j) dma_one(vrsrc, vstride, voffs, kv0, j, vslot(slot));
  };
  // first token of tile t, clamped to the task's tiles
  auto tile_kv0 = [&](int t) -> int { return kvt[t < 0 ? 0 : t < nkv_tiles ? t : nkv_tiles - 1] * TKV; };

  // lane-constant LDS offsets
  const int sw = swz(lane & 15);
  int koff[8];  // K operand: row (lane % 32) of a 32-key block, chunk 2c + hh
#pragma unroll
  for (int c = 0; c < 8; ++c) koff[c] = (lane & 31) * kRowBytes + (((2 * c + hh) ^ sw) << 4);
  int voff[2][4];  // V transposed read: [r][dblk]
  {
    const int s16 = lane & 15, gi = lane >> 4, mh = gi & 1, gh = gi >> 1;
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

  // membership decode for this lane's query rows
  int mem_row[G];
#pragma unroll
  for (int g = 0; g < G; ++g) mem_row[g] = (a.gq > 1) ? (q_local(g) >> a.bq_shift) : 0;
  const int mem_bits = a.gq * a.gkv;
  const uint64_t full = (mem_bits >= 64) ? ~0ull : ((1ull << mem_bits) - 1);
  // membership bits of tile t: the plan's bitmap, or, for plans that record
  // none, the zero page inverted (every member active); no branch, so the
  // scalar loads of one iteration issue together
  const cu64p mbits = a.member ? (cu64p)(a.member + tb) : (cu64p)a.zero_page;
  const int mstep = a.member ? 1 : 0;
  const uint64_t minv = a.member ? 0ull : ~0ull;
  auto bits_of = [&](int t) -> uint64_t { return (mbits[t * mstep] ^ minv) & full; };
  const bf16x2 ones2 = {(__bf16)1.0f, (__bf16)1.0f};

  f32x16 o[G][4];
#pragma unroll
  for (int g = 0; g < G; ++g) {
#pragma unroll
    for (int i = 0; i < 4; ++i) o[g][i] = f32x16{};
  }
  float m_run[G], l_run[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m_run[g] = kNegInf;
    l_run[g] = 0.f;
  }

  // MFMA operand stream of one iteration: units [0, kNA) are the S^T MFMAs of
  // the next tile (A = K rows), units [kNA, kNU) the O^T MFMAs of this tile
  // (A = V^T via transposed reads); each unit issues one MFMA per row group
  // with the same A operand.  Operands are read kAhead units ahead.
  constexpr int kNA = 8 * kNKB;
  constexpr int kNB = 4 * (TKV / 16);
  constexpr int kNU = kNA + kNB;
  auto load_op = [&](int u, const uint8_t* ks, const uint8_t* vs) -> bf16x8 {
    if (u < kNA) {
      const int c = u / kNKB, kb = u % kNKB;
      return *reinterpret_cast<const bf16x8*>(ks + kb * 32 * kRowBytes + koff[c]);
    }
    const int j = u - kNA, t = j / 4, dblk = j % 4;
    const i16x4 lo = lds_read_tr(vs + t * 16 * kRowBytes + voff[0][dblk]);
    const i16x4 hi = lds_read_tr(vs + t * 16 * kRowBytes + voff[1][dblk]);
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  };

  // Score and probability registers of one tile are indexed [g * kNKB + kb]
  // (score blocks) and [g * kChunks + c] (packed bf16 P chunks).
  constexpr int kE = 16 * kNKB;           // score elements per lane and group
  constexpr int kChunks = TKV / 16;       // 8-element P chunks per group

  // raw scores S^T of one tile with nothing else to overlap (prologue)
  auto qk_only = [&](const uint8_t* ks, f32x16* s) {
#pragma unroll
    for (int i = 0; i < G * kNKB; ++i) s[i] = f32x16{};
    bf16x8 op[3];
    op[0] = load_op(0, ks, nullptr);
    op[1] = load_op(1, ks, nullptr);
#pragma unroll
    for (int u = 0; u < kNA; ++u) {
      if (u + 2 < kNA) op[(u + 2) % 3] = load_op(u + 2, ks, nullptr);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        if constexpr (G == 1) s[g * kNKB + u % kNKB] = mfma32(op[u % 3], qf[g][u / kNKB], s[g * kNKB + u % kNKB]);
        else mfma32_vacc(s[g * kNKB + u % kNKB], op[u % 3], qf[g][u / kNKB], u < kNKB);
      }
    }
  };

  // entries outside the tile's active members or past the sequence end ->
  // -inf; returns whether this lane's row keeps any key of the tile
  auto apply_mask = [&](f32x16* s, int kv0, uint64_t bits, int mrow) -> bool {
    const uint64_t rowbits = bits >> (mrow * a.gkv);
    // allowed-key bitmap of this lane's row over the tile
    uint64_t allowed = 0;
    const int nvalid = min(TKV, a.Nkv - kv0);
    const uint64_t tailmask = nvalid >= 64 ? ~0ull : ((1ull << nvalid) - 1);
    if (a.gkv > 1) {
      const int bkv = 1 << a.bkv_shift;
      const uint64_t run = bkv >= 64 ? ~0ull : ((1ull << bkv) - 1);
      for (int cm = 0; cm < a.gkv; ++cm)
        if ((rowbits >> cm) & 1ull) allowed |= run << (cm * bkv);
    } else {
      allowed = (rowbits & 1ull) ? ~0ull : 0ull;
    }
    allowed &= tailmask;
    const uint64_t mine = allowed >> (4 * hh);
#pragma unroll
    for (int kb = 0; kb < kNKB; ++kb) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int jc = kb * 32 + (i >> 2) * 8 + (i & 3);  // key index minus 4 * hh
        float x = s[kb][i];
        mask_inplace(x, (mine >> jc) & 1ull);
        s[kb][i] = x;
      }
    }
    return allowed != 0;
  };

  // Row maximum of one group's raw scores in a tile (the scale is positive),
  // both lane halves combined.
  auto row_max = [&](const f32x16* s) -> float {
    float mx = kNegInf;
#pragma unroll
    for (int kb = 0; kb < kNKB; ++kb) {
#pragma unroll
      for (int i = 0; i < 16; i += 2) mx = fmaxf(mx, fmaxf(s[kb][i], s[kb][i + 1]));
    }
    return fmaxf(mx, other_half(mx));
  };

  // Distribution of the VALU work of one iteration over its MFMAs.
  // A probability is made in two steps one slot apart: the exponential
  // (stage A) and, for a pair of them, the bf16 packing and the row-sum dot
  // product (stage B), so no slot waits on an exponential it just issued.
  // Stage A is spread over all but the last slot; none of it feeds an MFMA
  // of the same iteration.
  constexpr int kEAll = G * kE;           // score elements per lane, all groups
  constexpr int kGroupLoads = 2 * kLoadsPerWave;  // refill loads of one iteration
  // Refill loads go out one every kDmaEvery units.  The T_Q = 64 kernels run
  // one wave per SIMD, so no other workgroup covers a load still in flight
  // at the barrier: they issue the whole refill at the start of the
  // iteration (the slot it fills was released by the previous barrier).
  // With two workgroups per CU, spreading the loads measured faster.
  constexpr int kDmaEvery = NWAVES == 2 ? 1 : kNU / kGroupLoads;
  static_assert(kDmaEvery >= 1 && kDmaEvery * kGroupLoads <= kNU, "refill loads must fit the units");
  constexpr int kNS = kNU * G;            // MFMA slots of one iteration
  // elements whose exponential is formed by the end of slot ss
  auto a_end = [&](int ss) -> int { return ss < 0 ? 0 : ss < kNS - 1 ? (ss + 1) * kEAll / (kNS - 1) : kEAll; };
  constexpr int kAhead = 3;  // operand read distance, in units

  // probability of a raw score against the reference -nm, and the bf16
  // packing of a pair of them (register k of chunk c holds elements 8c + 2k
  // and 8c + 2k + 1)
  auto exponent = [&](float sv, float nm) { return fast_exp2(__builtin_fmaf(sv, c_log2, nm)); };
  auto pack_pair = [&](float p0, float p1) { return __builtin_convertvector((f32x2){p0, p1}, bf16x2); };

  // One pipeline iteration over tile t: (rare) masking of s_cur; the S^T
  // MFMAs of tile t+1 (K from ks_next) and the O^T MFMAs of tile t-1 (V from
  // vs_prev, P from pw_prev) interleaved with the probabilities of tile t
  // (into pw_cur).  Leaves each group's lane sum of those probabilities in
  // lsum; active tells whether the lane's row of a group has a key in tile t.
  auto iteration = [&](f32x16* s_cur, f32x16* s_nxt, int kv0_cur, uint64_t bits_cur, const uint8_t* ks_next,
                       const uint8_t* vs_prev, u32x4* pw_cur, const u32x4* pw_prev, int kv0_refill_k,
                       int kv0_refill_v, uint8_t* k_refill, uint8_t* v_refill, bool* active, float* lsum) {
    // the ring refill of this iteration goes out one load every kDmaEvery units
#pragma unroll
    for (int g = 0; g < G; ++g) active[g] = true;
    if (__builtin_expect(kv0_cur + TKV > a.Nkv || bits_cur != full, 0)) {
#pragma unroll
      for (int g = 0; g < G; ++g) active[g] = apply_mask(s_cur + g * kNKB, kv0_cur, bits_cur, mem_row[g]);
    }
    float nm[G];
#pragma unroll
    for (int g = 0; g < G; ++g) nm[g] = (m_run[g] == kNegInf) ? 0.f : -m_run[g];
    float ls[G][2];
#pragma unroll
    for (int g = 0; g < G; ++g) ls[g][0] = ls[g][1] = 0.f;
    float pf[kEAll];
    auto stage_a = [&](int ei) {
      const int g = ei / kE, e = ei % kE;
      pf[ei] = exponent(s_cur[g * kNKB + e / 16][e % 16], nm[g]);
    };
    auto stage_b = [&](int pr) {
      const int e0 = 2 * pr, g = e0 / kE, el = e0 % kE;
      const bf16x2 pair = pack_pair(pf[e0], pf[e0 + 1]);
      pw_cur[g * kChunks + el / 8][(el % 8) / 2] = __builtin_bit_cast(uint32_t, pair);
      float& acc = ls[g][pr & 1];
      acc = __builtin_amdgcn_fdot2_f32_bf16(pair, ones2, acc, false);
      // keep the sum in this unit (otherwise it is sunk to the end of the loop)
      asm volatile("" : "+v"(acc));
    };
    bf16x8 op[kAhead + 1];
#pragma unroll
    for (int u = 0; u < kAhead; ++u) op[u] = load_op(u, ks_next, vs_prev);
    // one MFMA per slot: slot sl is row group sl % G of unit sl / G, so the
    // VALU work between two MFMAs of the wave stays short
#pragma unroll
    for (int sl = 0; sl < kNS; ++sl) {
      const int u = sl / G, g = sl % G;
      if (g == 0) {
        if (u + kAhead < kNU) op[(u + kAhead) % (kAhead + 1)] = load_op(u + kAhead, ks_next, vs_prev);
        if (u % kDmaEvery == 0 && u / kDmaEvery < kGroupLoads) {
          const int i = u / kDmaEvery;
          if (i < kLoadsPerWave) dma_one(krsrc, kstride, koffs, kv0_refill_k, i, k_refill);
          else dma_one(vrsrc, vstride, voffs, kv0_refill_v, i - kLoadsPerWave, v_refill);
        }
      }
      if (u < kNA) {
        f32x16& acc = s_nxt[g * kNKB + u % kNKB];
        if constexpr (G == 1) {
          acc = mfma32(op[u % (kAhead + 1)], qf[g][u / kNKB], u < kNKB ? f32x16{} : acc);
        } else {
          mfma32_vacc(acc, op[u % (kAhead + 1)], qf[g][u / kNKB], u < kNKB);
        }
      } else {
        const int j = u - kNA;
        o[g][j % 4] = mfma32(op[u % (kAhead + 1)], __builtin_bit_cast(bf16x8, pw_prev[g * kChunks + j / 4]),
                             o[g][j % 4]);
      }
#pragma unroll
      for (int pr = a_end(sl - 2) / 2; pr < a_end(sl - 1) / 2; ++pr) stage_b(pr);
#pragma unroll
      for (int e = a_end(sl - 1); e < a_end(sl); ++e) stage_a(e);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int g = 0; g < G; ++g) lsum[g] = ls[g][0] + ls[g][1];
  };

  // Rare path after an iteration, for row group g: in the rows flagged by
  // `mine` (both lane halves of a row agree) a probability of tile t may
  // exceed 2^8, or the row met its first key.  Raise those rows' reference
  // to the maximum of their scores so far, rescale their O and l, and form
  // the tile's probabilities again.  O holds P V up to tile t-1, all against
  // the old reference, so one factor per row covers it.  Other rows keep
  // their state exactly: their factor is 1 and their probabilities are
  // formed again from the same operands, which gives the same bits.
  auto raise_reference = [&](int g, const f32x16* s_cur, u32x4* pw_cur, bool mine, float lsum_old) -> float {
    const float mxs = row_max(s_cur + g * kNKB) * c_log2;
    const float m_new = mine ? fmaxf(m_run[g], mxs) : m_run[g];
    const float alpha = (m_new == m_run[g]) ? 1.f : fast_exp2(m_run[g] - m_new);
    m_run[g] = m_new;
    l_run[g] *= alpha;
#pragma unroll
    for (int d = 0; d < 4; ++d) scale_inplace<G == 1>(o[g][d], alpha);
    const float nm = (m_run[g] == kNegInf) ? 0.f : -m_run[g];
    float ls = 0.f;
#pragma unroll
    for (int pr = 0; pr < kE / 2; ++pr) {
      const int e0 = 2 * pr;
      const bf16x2 pair = pack_pair(exponent(s_cur[g * kNKB + e0 / 16][e0 % 16], nm),
                                    exponent(s_cur[g * kNKB + e0 / 16][e0 % 16 + 1], nm));
      pw_cur[g * kChunks + e0 / 8][(e0 % 8) / 2] = __builtin_bit_cast(uint32_t, pair);
      ls = __builtin_amdgcn_fdot2_f32_bf16(pair, ones2, ls, false);
    }
    return mine ? ls : lsum_old;
  };

  // number of DMA instructions one iteration issues (K tile and V tile)
  constexpr int kGroup = 2 * kLoadsPerWave;
  constexpr int kInFlight = (STAGES - 2) * kGroup;

  f32x16 sA[G * kNKB], sB[G * kNKB];
  u32x4 pwA[G * kChunks], pwB[G * kChunks];
#pragma unroll
  for (int c = 0; c < G * kChunks; ++c) pwB[c] = u32x4{};  // P of "tile -1": no contribution
  // scalars for the coming iteration, fetched one iteration ahead
  int kv_next_k = 0, kv_next_v = 0, kv_cur = 0;
  uint64_t bits_cur = full;
  if (nkv_tiles > 0) {
    // prologue: K of tile 0 into slot 0, then slot j <- (K of tile j, V of
    // tile j-2) for j = 1..STAGES-1, in the order they are needed (V of the
    // "tile -1" that iteration 0 multiplies by zero probabilities is tile 0,
    // any finite data).  Ring refills are never skipped: past the end of the
    // task they re-load its last tile into the free slot, which keeps the
    // count of loads in flight the same on every path.
    dma_k(tile_kv0(0), 0);
#pragma unroll
    for (int j = 1; j < STAGES; ++j) {
      dma_k(tile_kv0(j), j);
      dma_v(tile_kv0(j - 2), j);
    }
    kv_next_k = tile_kv0(STAGES);
    kv_next_v = tile_kv0(STAGES - 2);
    kv_cur = tile_kv0(0);
    bits_cur = bits_of(0);
    // the scores of tile 0 need K0 only
    wait_vm_lgkm<(STAGES - 1) * kGroup>();
    block_sync();
    if constexpr (G > 1) hazard_wait_q2(qf);
    qk_only(kslot(0), sA);
    if constexpr (G > 1) {
#pragma unroll
      for (int i = 0; i < G * kNKB; ++i) hazard_wait_v(sA[i]);
    }
    // the first iteration needs slot 1
    wait_vm_lgkm<kInFlight>();
    block_sync();  // every wave has read slot 0 before it is refilled
  }
  for (int t0 = 0; t0 < nkv_tiles; t0 += STAGES) {
#pragma unroll
    for (int u = 0; u < STAGES; ++u) {
      const int t = t0 + u;
      if (t >= nkv_tiles) break;
      // refill slot t % STAGES with K of tile t+STAGES and V of tile
      // t+STAGES-2 (issued inside the iteration, spread over its MFMA units)
      f32x16* s_cur = (u % 2 == 0) ? sA : sB;
      f32x16* s_nxt = (u % 2 == 0) ? sB : sA;
      u32x4* pw_cur = (u % 2 == 0) ? pwA : pwB;
      u32x4* pw_prev = (u % 2 == 0) ? pwB : pwA;
      bool active[G];
      float lsum[G];
      iteration(s_cur, s_nxt, kv_cur, bits_cur, kslot((u + 1) % STAGES), vslot((u + 1) % STAGES), pw_cur, pw_prev,
                kv_next_k, kv_next_v, kslot(u), vslot(u), active, lsum);
      // the check of tile t before any MFMA uses its probabilities (sums of
      // probabilities in [0, inf] are never NaN)
      auto needs_raise = [&](int g) { return lsum[g] > kSumMax || (m_run[g] == kNegInf && active[g]); };
      uint64_t need_any = 0;
#pragma unroll
      for (int g = 0; g < G; ++g) need_any |= __ballot(needs_raise(g));
      if (__builtin_expect(need_any != 0, 0)) {
#pragma unroll
        for (int g = 0; g < G; ++g) {
          // both lane halves of a row take the same decision; the exchange
          // runs in every lane (under a short-circuit || it would run only in
          // some lanes, and a lane swap there reads inactive partners)
          const uint32_t mine = needs_raise(g) ? 1u : 0u;
          const bool row = (mine | other_half_u32(mine)) != 0;
          if (__ballot(row) != 0) lsum[g] = raise_reference(g, s_cur, pw_cur, row, lsum[g]);
        }
      }
#pragma unroll
      for (int g = 0; g < G; ++g) l_run[g] += lsum[g];
      // scalars of the next iteration, complete before the barrier so no
      // scalar load is outstanding while the next iteration's LDS reads are
      // counted
      kv_next_k = tile_kv0(t + 1 + STAGES);
      kv_next_v = tile_kv0(t + STAGES - 1);
      kv_cur = tile_kv0(t + 1);
      bits_cur = bits_of(t + 1 < nkv_tiles ? t + 1 : nkv_tiles - 1);
      asm volatile("" ::"s"(kv_next_k), "s"(kv_next_v), "s"(kv_cur), "s"(bits_cur));
      // slot (t+2) % STAGES must have landed; younger loads may fly
      wait_vm_lgkm<kInFlight>();
      block_sync();
    }
  }
  if (nkv_tiles > 0) {
    // O += P V of the last tile n-1: its V sits in slot (n+1) % STAGES
    const u32x4* pw_last = ((nkv_tiles - 1) % 2 == 0) ? pwA : pwB;
    const int sl = (nkv_tiles + 1) % STAGES;
    const uint8_t* vs_last = vslot(sl);
    bf16x8 vop[2];
    vop[0] = load_op(kNA, nullptr, vs_last);
#pragma unroll
    for (int j = 0; j < kNB; ++j) {
      if (j + 1 < kNB) vop[(j + 1) % 2] = load_op(kNA + j + 1, nullptr, vs_last);
#pragma unroll
      for (int g = 0; g < G; ++g)
        o[g][j % 4] = mfma32(vop[j % 2], __builtin_bit_cast(bf16x8, pw_last[g * kChunks + j / 4]), o[g][j % 4]);
    }
  }
  // no load of this workgroup may still be writing LDS when it ends
  wait_vm_lgkm<0>();

  // ---- epilogue
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const float l_tot = l_run[g] + other_half(l_run[g]);
    const int ql = q_local(g), qr = q_row(g);
    if (task.nsplit == 1) {
      if (qr < a.Nq) {
        const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
        uint16_t* op = a.o + b * a.os0 + h * a.os1 + (int64_t)qr * a.os2;
#pragma unroll
        for (int dblk = 0; dblk < 4; ++dblk) {
#pragma unroll
          for (int gg = 0; gg < 4; ++gg) {
            bf16x4 v4;
#pragma unroll
            for (int e = 0; e < 4; ++e) v4[e] = (__bf16)(o[g][dblk][4 * gg + e] * inv);
            *reinterpret_cast<bf16x4*>(op + dblk * 32 + 8 * gg + 4 * hh) = v4;
          }
        }
        if (a.lse && hh == 0) {
          a.lse[((int64_t)b * a.H + h) * a.Nq + qr] =
              l_tot > 0.f ? (m_run[g] + __log2f(l_tot)) * 0.69314718055994530942f : kNegInf;
        }
      }
    } else {
      // Split-K partial state: reference m (log2 domain), l, O unnormalised
      float* slot = a.ws + ti * (int64_t)C::kTQ * (kD + 2);
      if (hh == 0) {
        slot[ql] = l_tot > 0.f ? m_run[g] : kNegInf;
        slot[C::kTQ + ql] = l_tot;
      }
      float* os = slot + 2 * C::kTQ + (int64_t)ql * kD;
#pragma unroll
      for (int dblk = 0; dblk < 4; ++dblk) {
#pragma unroll
        for (int gg = 0; gg < 4; ++gg) {
          f32x4 v4;
#pragma unroll
          for (int e = 0; e < 4; ++e) v4[e] = o[g][dblk][4 * gg + e];
          *reinterpret_cast<f32x4*>(os + dblk * 32 + 8 * gg + 4 * hh) = v4;
        }
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

template <int NWAVES, int G, int TKV, int STAGES>
hipError_t launch_variant(const AttnArgs& a, hipStream_t s) {
  const int64_t slots = a.nslots > 0 ? a.nslots : default_slots(a.ntasks);
  if (slots == 0) return hipSuccess;
  hipLaunchKernelGGL((attn_fwd_kernel<NWAVES, G, TKV, STAGES>), dim3((unsigned)slots), dim3(64 * NWAVES), 0, s, a);
  return hipGetLastError();
}

}  // namespace

// The kernel of a catalog entry: physical tile, wavefronts per workgroup and
// ring depth (Section 4.4).  With two waves per SIMD a workgroup may use
// 64 KB of LDS (two per CU): four slots of 32-key tiles or two of 64-key
// tiles.  T_Q = 256 with 32-key tiles runs four waves of 64 rows (two row
// groups sharing every K and V operand, one workgroup per CU, eight slots);
// with 64-key tiles eight waves of 32 rows.
hipError_t launch_attention(int tq, int tkv, int waves, int stages, const AttnArgs& a, hipStream_t s) {
  if (tq == 64 && tkv == 32 && waves == 2 && stages == 4) return launch_variant<2, 1, 32, 4>(a, s);
  if (tq == 64 && tkv == 32 && waves == 2 && stages == 2) return launch_variant<2, 1, 32, 2>(a, s);
  if (tq == 64 && tkv == 64 && waves == 2 && stages == 2) return launch_variant<2, 1, 64, 2>(a, s);
  if (tq == 128 && tkv == 32 && waves == 4 && stages == 4) return launch_variant<4, 1, 32, 4>(a, s);
  if (tq == 128 && tkv == 32 && waves == 4 && stages == 2) return launch_variant<4, 1, 32, 2>(a, s);
  if (tq == 128 && tkv == 64 && waves == 4 && stages == 2) return launch_variant<4, 1, 64, 2>(a, s);
  if (tq == 256 && tkv == 32 && waves == 4 && stages == 8) return launch_variant<4, 2, 32, 8>(a, s);
  if (tq == 256 && tkv == 64 && waves == 8 && stages == 2) return launch_variant<8, 1, 64, 2>(a, s);
  if (tq == 256 && tkv == 64 && waves == 8 && stages == 4) return launch_variant<8, 1, 64, 4>(a, s);
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
