// Fused residual workload predictor for gfx950 (MI355X).
//
// One kernel computes, for a tile of tokens, the early router logits (Sec. "Residual Workload
// Prediction", Eq. 2 with the linear router of Eq. 4), the routed model's scores and its
// (optionally group-limited) top-k selection, and the per-expert token histogram of Eq. 5.  The
// last workgroup to finish folds the histogram into per-rank loads under the expert-to-rank
// placement (Alg. 1, second step) and computes the max-to-mean ratio (Sec. "Metrics").
//
// Workgroup: 4 waves (256 threads), one per SIMD, one workgroup per CU.  A wave may then hold up to
// 512 registers, which the contraction spends on deep prefetching rather than on extra waves:
//   * Hidden rows go from HBM straight into LDS (buffer_load ... lds, 16 bytes per lane): no
//     register round trip and no LDS store instructions.  The k dimension runs in stages of 256
//     bytes of every row; a ring of NS stage buffers keeps up to NS - 1 stages in flight beyond the
//     one being read.  Each
//     workgroup-wide load instruction writes 4 rows x 256 bytes; inside a row the 16-byte chunks are
//     XOR-swizzled by the row index so the fragment reads below are free of bank conflicts.
//   * Each wave owns a slice of the experts (and, for small E, of the tokens).  Its router-weight
//     fragments come from the pre-packed weight (one contiguous 1 KB per load instruction,
//     L2-resident) straight into registers through a ring of 16 k-step slices, 15 k-steps ahead of
//     the MFMAs; the hidden fragments are read from LDS one k-step ahead.  The router weight is the
//     A operand (M = experts) and the hidden tile is B (N = tokens): v_mfma_f32_32x32x16_bf16 (or
//     32x32x2 f32), so each lane ends with groups of four consecutive experts of one token.
//   * One workgroup barrier per stage, placed before the stage's last k-step: it publishes the next
//     stage (every wave waits for its own share of that stage's loads first) and frees the buffer
//     just read, which the next load batch then refills.  Waits are counted, never drained.
// The logits never leave the chip: scores go to an LDS tile, EPAD/32 lanes cooperate on one
// token, and the histogram is privatised in LDS with one global atomic per expert per workgroup.
//
// Selection is exact in float32 with ties to the lower expert index.  The fast path ranks 32-bit
// keys (top 24 bits of the order-preserving score encoding, then 255 - expert); its set equals the
// exact top-k whenever the k-th and (k+1)-th keys differ in their score bits, and tokens where they
// do not take an exact 64-bit path.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>
#include <type_traits>

#include "fb_internal.h"
#include "fb_plan_wave.h"

namespace fb {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr;

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kStepBytes = 32;                  // bytes of a row feeding one MFMA k-step
constexpr int kNStep = 8;                       // k-steps per stage
constexpr int kStageRowBytes = kStepBytes * kNStep;   // 256
constexpr int kRingW = 16;                      // router-weight k-step slices held per wave
constexpr int kMaxK = FB_MAX_TOPK;
constexpr int kMaxGroups = 32;
constexpr uint32_t kRsrcWord3 = 0x00020000u;    // raw buffer, 32-bit dwords
constexpr uint32_t kOobOffset = 0x80000000u;    // fails the buffer range check: load returns 0
#ifndef FB_SEL_CACHE
#define FB_SEL_CACHE 7
#endif
constexpr int kCache = FB_SEL_CACHE;            // per-lane cached keys in the top-k extraction

// Tile shapes: WE waves along experts x WT waves along tokens, BM tokens per workgroup; every wave
// tile is a whole number of 32 x 32 MFMA blocks.
template <int EPAD> struct TileCfg;
template <> struct TileCfg<256> { static constexpr int WE = 4, WT = 1, BM = 128; };
template <> struct TileCfg<128> { static constexpr int WE = 4, WT = 1, BM = 64; };
template <> struct TileCfg<64> { static constexpr int WE = 2, WT = 2, BM = 64; };
template <> struct TileCfg<32> { static constexpr int WE = 1, WT = 4, BM = 128; };

// Stages of the LDS ring for a tile height.  Each wave may have at most 63 vector-memory loads in
// flight; NS is the deepest ring whose counted waits stay below that (checked in the kernel).
constexpr int ring_stages(int BM) { return BM >= 128 ? 3 : 4; }

struct Params {
  const char* x;
  int64_t T;
  int32_t Hbytes;
  int32_t ldx_bytes;
  const char* wpack;   // packed router weight (see pack_kernel)
  int32_t E;
  const float* logit_bias;
  const float* select_bias;
  int32_t kind, k, n_group, topk_group, group_topn;
  const int32_t* e2r;
  int32_t R;
  int32_t* counts;
  int32_t* rank_loads;
  double* max_mean;
  int32_t* ws_acc;
  uint32_t* ws_ticket;
  uint32_t* ws_tile;   // split mode: arrivals per tile (kSplit)
  int32_t* topk_idx;
  float* logits;
  uint32_t nblocks;
  int32_t nstages;     // stages this workgroup contracts
  int32_t st_base;     // first of them
  int32_t st_total;    // stages of a whole row
  int32_t ks;          // splits of the stage range (split mode); 1 otherwise
  float* partial;      // split mode: partial logits, [tile][split][register][thread]
  int32_t plan_cpl;    // 0: no plan; 1 or 2: the one-wave planner's candidates per lane
  PlanDeviceLaunch plan;   // the swap plan of the counts, made by the last workgroup
};

// Workgroup barrier that orders LDS only; outstanding global loads stay in flight across it.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
}

// 32-bit LDS address of a pointer into a __shared__ array.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// 16-byte LDS read as an instruction of its own; its completion is awaited with lgkm_wait.
__device__ __forceinline__ void ds_read_b128(u32x4& dst, uint32_t addr, int offset) {
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(dst) : "v"(addr), "i"(offset));
}
template <int N>
__device__ __forceinline__ void lgkm_wait() {
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N));
}
template <int N>
__device__ __forceinline__ void vm_wait() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N));
}
// 16-byte buffer load into accumulation registers, as an instruction of its own; its completion is
// awaited with vm_wait.  rsrc: buffer descriptor (base, num_records bytes, raw 32-bit words).
__device__ __forceinline__ void buffer_load_b128_acc(u32x4& dst, const i32x4& rsrc, uint32_t voff,
                                                     uint32_t soff) {
  asm volatile("buffer_load_dwordx4 %0, %1, %2, %3 offen" : "=a"(dst) : "v"(voff), "s"(rsrc), "s"(soff));
}
// After an explicit wait: the values below are (re)defined here, so nothing reads them earlier.
template <int N>
__device__ __forceinline__ void pin(u32x4 (&v)[N]) {
#pragma unroll
  for (int i = 0; i < N; ++i) asm volatile("" : "+v"(v[i]));
}
template <int N>
__device__ __forceinline__ void pin_acc(u32x4 (&v)[N]) {
#pragma unroll
  for (int i = 0; i < N; ++i) asm volatile("" : "+a"(v[i]));
}

// s_waitcnt immediate: at most `vm` vector-memory loads outstanding (6-bit count) and at most `lgkm`
// LDS/scalar operations (expcnt left free).
constexpr int waitcnt_imm(int vm, int lgkm) {
  return (vm & 15) | (((vm >> 4) & 3) << 14) | (7 << 4) | ((lgkm & 15) << 8);
}

// Order-preserving map of float bits to unsigned (for finite values; -0 is canonicalised first).
__device__ __forceinline__ uint32_t ord_bits(float s) {
  const uint32_t u = __float_as_uint(s);
  return u ^ ((uint32_t)((int32_t)u >> 31) | 0x80000000u);
}

// Inverse of ord_bits.
__device__ __forceinline__ float from_ord_bits(uint32_t o) {
  return __uint_as_float((o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o);
}

// Median of three (v_med3_u32): the middle value, used to maintain a sorted top-3.
__device__ __forceinline__ uint32_t umed3(uint32_t a, uint32_t b, uint32_t c) {
  return max(min(a, b), min(max(a, b), c));
}

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// DPP patterns that stay inside aligned groups of 2, 4, 8 and 16 lanes.
constexpr int kXor1 = 0xB1;       // quad_perm [1,0,3,2]
constexpr int kXor2 = 0x4E;       // quad_perm [2,3,0,1]
constexpr int kXor3 = 0x1B;       // quad_perm [3,2,1,0]
constexpr int kHalfMirror = 0x141;
constexpr int kMirror = 0x140;

// Maximum of v over the aligned group of G lanes containing this lane.
template <int G>
__device__ __forceinline__ uint32_t group_max_u32(uint32_t v) {
  if constexpr (G >= 2) v = max(v, dpp_u32<kXor1>(v));
  if constexpr (G >= 4) v = max(v, dpp_u32<kXor2>(v));
  if constexpr (G >= 8) v = max(v, dpp_u32<kHalfMirror>(v));
  if constexpr (G >= 16) v = max(v, dpp_u32<kMirror>(v));
  return v;
}

// Merge (m1 >= m2) pairs across the aligned group of g lanes (g a power of two <= 16).
template <int CTRL>
__device__ __forceinline__ void top2_merge_step(float& m1, float& m2) {
  const float o1 = dpp_f32<CTRL>(m1), o2 = dpp_f32<CTRL>(m2);
  const float hi = fmaxf(m1, o1), lo = fminf(m1, o1);
  m2 = fmaxf(lo, fmaxf(m2, o2));
  m1 = hi;
}
__device__ __forceinline__ void top2_group(float& m1, float& m2, int g) {
  if (g >= 2) top2_merge_step<kXor1>(m1, m2);
  if (g >= 4) top2_merge_step<kXor2>(m1, m2);
  if (g >= 8) top2_merge_step<kHalfMirror>(m1, m2);
  if (g >= 16) top2_merge_step<kMirror>(m1, m2);
}

// Rank of this lane's group among the groups of its token (score desc, lower group first), for
// groups that each cover lpg whole lanes of the token's G lanes (lane jl covers experts 32 jl ..
// 32 jl + 31; lanes at or past E hold no group).  Values of the other lanes of the aligned
// G-lane group come in by lane exchange: lanes jl ^ 1..3 through quad permutations, lanes
// jl ^ 4..7 through the half-row mirror (lane jl ^ 7) followed by the same permutations.
// Which lanes jl ^ x lead a group (lead[x]) and whose group comes before this lane's (lower[x]) does
// not depend on the token: computed once, as 0/1 integers kept in vector registers, so the rank is
// plain compare-and-select arithmetic with no branches.
template <int G>
struct RankLanes { int lead[G], lower[G]; };
template <int G>
__device__ __forceinline__ RankLanes<G> rank_lanes(int jl, int lpg, int E) {
  RankLanes<G> r;
  const int me = jl / lpg;
#pragma unroll
  for (int x = 0; x < G; ++x) {
    const int j = jl ^ x;
    r.lead[x] = (x != 0 && (j % lpg) == 0 && j * 32 < E) ? 1 : 0;
    r.lower[x] = (j / lpg < me) ? 1 : 0;
    asm volatile("" : "+v"(r.lead[x]), "+v"(r.lower[x]));
  }
  return r;
}
template <int G>
__device__ __forceinline__ int group_rank(float g, const RankLanes<G>& rl) {
  float v[8];
  v[0] = g;
  if constexpr (G >= 2) v[1] = dpp_f32<kXor1>(g);
  if constexpr (G >= 4) { v[2] = dpp_f32<kXor2>(g); v[3] = dpp_f32<kXor3>(g); }
  if constexpr (G >= 8) {
    const float m = dpp_f32<kHalfMirror>(g);   // lane jl ^ 7
    v[7] = m; v[6] = dpp_f32<kXor1>(m); v[5] = dpp_f32<kXor2>(m); v[4] = dpp_f32<kXor3>(m);
  }
  int rank = 0;
#pragma unroll
  for (int x = 1; x < G; ++x) {
    const float o = v[x];
    const int gt = o > g ? 1 : 0, eq = o == g ? 1 : 0;
    rank += rl.lead[x] & (gt | (eq & rl.lower[x]));
  }
  return rank;
}

// ---- packed router weight --------------------------------------------------------------------
// Stage st (kStageRowBytes of every row) occupies EPAD * kStageRowBytes contiguous bytes.  Inside
// it, the 1 KB chunk c = (we * kNStep + q) * FE + fe holds, for lane l, the 16 bytes of row
// e = we * EW + fe * 32 + (l & 31) at byte st * kStageRowBytes + q * 32 + (l >> 5) * 16 of that row:
// exactly the A-operand fragment wave `we` loads for expert block fe of k-step q.  Rows >= E and
// bytes past H are zero.
template <int EPAD>
__global__ void pack_kernel(const char* __restrict__ w, int32_t E, int32_t Hbytes, int32_t nstages,
                            u32x4* __restrict__ out) {
  using Cfg = TileCfg<EPAD>;
  constexpr int EW = EPAD / Cfg::WE, FE = EW / 32;
  constexpr int kUnitsPerStage = EPAD * (kStageRowBytes / 16);   // 16-byte units
  const int64_t units = (int64_t)nstages * kUnitsPerStage;
  for (int64_t idx = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; idx < units;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int st = (int)(idx / kUnitsPerStage);
    const int rem = (int)(idx % kUnitsPerStage);
    const int c = rem >> 6, l = rem & 63;
    const int fe = c % FE, q = (c / FE) % kNStep, we = c / (FE * kNStep);
    const int e = we * EW + fe * 32 + (l & 31);
    const int b = st * kStageRowBytes + q * kStepBytes + (l >> 5) * 16;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (e < E && b < Hbytes) v = *reinterpret_cast<const u32x4*>(w + (int64_t)e * Hbytes + b);
    out[idx] = v;
  }
}

// ---- the contraction ---------------------------------------------------------------------------
// acc[fe][ft] += (router weight block fe) x (hidden block ft) over every stage of the tile; the NS
// stage buffers start at ring_lds.
template <bool BF16, int EPAD, int FE, int FT, int NS, int BM, int TW>
__device__ __forceinline__ void contract(f32x16 (&acc)[FE][FT], const Params& p, int64_t row0,
                                         int wave, int we, int wt, int lane, char* ring_lds) {
  constexpr int LPW = BM / 4 / kWaves;               // stage load instructions per wave (4 rows each)
  constexpr int UNROLL = kRingW / kNStep;            // one period of the weight ring per iteration
  constexpr int STAGE = BM * kStageRowBytes;         // LDS bytes of one stage buffer
  // counted waits (see the issue order below): loads issued after a stage's own batch by the time
  // the stage must be resident, and the most a wave ever has in flight
  constexpr int kWaitStage = 8 * FE * (NS - 1) + (NS - 2) * LPW;
  // the batch of stage t goes out at the end of stage t - NS, right before the weight slice of
  // k-step kLead + 8 t; the prologue keeps that order for stages 0 .. NS-1
  constexpr int kLead = kNStep - 1 + kRingW - 1 - kNStep * NS;
  static_assert(kLead < 0, "stage 0's batch precedes every weight slice");
  // Batches the prologue issues before any weight slice have fewer loads behind them than the
  // steady-state count assumes; the prologue waits for all of them (they went out together).
  constexpr int kEarly = (-kLead + kNStep - 1) / kNStep;          // stages t with kLead + 8 t < 0
  constexpr int kWaitFirst = (NS - kEarly) * LPW + (kRingW - 1) * FE;
  static_assert(kWaitStage <= 63 && (kRingW - 1) * FE + NS * LPW <= 63,
                "more loads in flight than a wave can count");
  static_assert(LPW >= 1 && BM % (4 * kWaves) == 0, "stage loads split evenly over the waves");
  static_assert(kRingW % kNStep == 0, "the weight ring holds whole stages");
  const uint32_t lds0 = lds_addr(ring_lds);
  const int nst = p.nstages;
  const int Hb = p.Hbytes;
  const int64_t rows = (p.T - row0) < BM ? (p.T - row0) : BM;

  // hidden rows: rows past T are outside the buffer and read as zero
  const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(p.x + row0 * (int64_t)p.ldx_bytes), (short)0, (int)(rows * p.ldx_bytes), kRsrcWord3);
  // Load instruction j of this wave fills rows 4 (wave LPW + j) + (lane >> 4); lane l writes the
  // 16-byte slot (l & 15) of its row, which holds logical chunk (l & 15) ^ (row & 15).
  uint32_t voff[LPW];
  int cbyte[LPW];
#pragma unroll
  for (int j = 0; j < LPW; ++j) {
    const int r = 4 * (wave * LPW + j) + (lane >> 4);
    const int c = (lane & 15) ^ (r & 15);
    voff[j] = (uint32_t)(r * p.ldx_bytes + c * 16);
    cbyte[j] = c * 16;
  }
  // a stage's batch; bytes at or past H (tail of the last stage) and stages past the end are not
  // fetched and land as zeros
  // The counted waits below assume each batch goes out whole, in program order with the weight
  // slices: the scheduling barriers keep other loads from moving into or across it.
  auto load_stage = [&](int bi, int st) {        // bi: stage buffer (wave-uniform)
    const bool live = st < nst;
    const int sb = live ? (p.st_base + st) * kStageRowBytes : 0;
    const int lim = live ? Hb - sb : 0;           // bytes of the stage inside the row (scalar)
    char* const dst = ring_lds + bi * STAGE + wave * LPW * 1024;
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < LPW; ++j) {
      const uint32_t off = cbyte[j] < lim ? voff[j] : kOobOffset;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_ptr)(dst + j * 1024), 16, off, sb, 0, 2);
    }
    __builtin_amdgcn_sched_barrier(0);
  };

  // router weight: stage st of the packed layout is EPAD * 256 bytes; this wave's fragment of
  // k-step q and expert block fe is the 1 KB chunk (we * kNStep + q) * FE + fe.  These loads are
  // instructions of their own (into accumulation registers, which the MFMAs read directly) with
  // counted waits: the issue order is fixed, so the count of loads issued after a k-step's slice is
  // known exactly, where the compiler's own tracking turns conservative at the loop head.
  constexpr int kPackStage = EPAD * kStageRowBytes;
  const uint64_t wbase_addr = reinterpret_cast<uint64_t>(p.wpack);
  const i32x4 wr = {(int32_t)(uint32_t)wbase_addr, (int32_t)(uint32_t)(wbase_addr >> 32),
                    p.st_total * kPackStage, (int32_t)kRsrcWord3};
  const uint32_t wbase = (uint32_t)(we * kNStep * FE * 1024 + lane * 16);
  auto load_w = [&](u32x4(&dst)[FE], int st, int q) {
    const bool ok = st < nst;
#pragma unroll
    for (int fe = 0; fe < FE; ++fe)
      buffer_load_b128_acc(dst[fe], wr, ok ? wbase + (uint32_t)((q * FE + fe) * 1024) : kOobOffset,
                           ok ? (p.st_base + st) * kPackStage : 0);
  };
  // loads issued after the weight slice of k-step q (of any stage) by the time its MFMAs start: the
  // slices of the next kRingW - 1 k-steps, and the stage batches issued at k-step 7 of the stages
  // in between (two of them, except for q = 6, whose window holds one)
  auto wait_w = [&](int q) {
    if (q == kNStep - 2) vm_wait<(kRingW - 1) * FE + LPW>();
    else vm_wait<(kRingW - 1) * FE + 2 * LPW>();
  };
  static_assert(kRingW - 1 > kNStep && kRingW - 1 < 2 * kNStep, "two stage batches per weight window");

  // hidden fragment of k-step q: token wt TW + ft 32 + (lane & 31), logical chunk 2q + (lane >> 5).
  // These LDS reads are written as instructions of their own, with their waits counted below: the
  // compiler cannot tell a read of one ring buffer from the stage loads still filling another and
  // would otherwise wait for every load in flight before each read.
  uint32_t baddr[kNStep];
#pragma unroll
  for (int q = 0; q < kNStep; ++q)
    baddr[q] = lds0 + (uint32_t)((wt * TW + (lane & 31)) * kStageRowBytes +
                                 (((2 * q + (lane >> 5)) ^ (lane & 15)) * 16));
  auto load_b = [&](u32x4(&dst)[FT], int bi, int q) {
    const uint32_t a = baddr[q] + (uint32_t)(bi * STAGE);
#pragma unroll
    for (int ft = 0; ft < FT; ++ft) ds_read_b128(dst[ft], a, ft * 32 * kStageRowBytes);
  };

  auto mma = [&](const u32x4(&a)[FE], const u32x4(&b)[FT]) {
#pragma unroll
    for (int ft = 0; ft < FT; ++ft) {
#pragma unroll
      for (int fe = 0; fe < FE; ++fe) {
        if constexpr (BF16) {
          acc[fe][ft] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8, a[fe]), __builtin_bit_cast(bf16x8, b[ft]), acc[fe][ft], 0, 0, 0);
        } else {
          // four k-pairs per fragment; A and B take the same k for every lane
          const f32x4 av = __builtin_bit_cast(f32x4, a[fe]);
          const f32x4 bv = __builtin_bit_cast(f32x4, b[ft]);
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc[fe][ft] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[j], bv[j], acc[fe][ft], 0, 0, 0);
        }
      }
    }
  };

  // ---- prologue: stages 0 .. NS-1 and k-steps 0 .. kRingW-2 in flight, then stage 0 published.
  // Loads go out in the steady state's order, so every wait at the loop head counts the same loads
  // on both paths into it.
  u32x4 ring[kRingW][FE];
  u32x4 bq[2][FT];
#pragma unroll
  for (int t = 0; t < NS; ++t)
    if (kLead + kNStep * t < 0) load_stage(t, t);
#pragma unroll
  for (int g = 0; g < kRingW - 1; ++g) {
#pragma unroll
    for (int t = 0; t < NS; ++t)
      if (kLead + kNStep * t == g) load_stage(t, t);
    load_w(ring[g], g / kNStep, g % kNStep);
    __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll
  for (int t = 0; t < NS; ++t)
    if (kLead + kNStep * t >= kRingW - 1) load_stage(t, t);
  __builtin_amdgcn_s_waitcnt(waitcnt_imm(kWaitFirst, 0));
  asm volatile("s_barrier" ::: "memory");
  load_b(bq[0], 0, 0);
  __builtin_amdgcn_sched_barrier(0);

  // ---- steady state.  Issue order per stage: k-steps 0..6 each read the next hidden fragments
  // and one weight slice; k-step 7 waits for this wave's share of stage s+1, meets the other waves
  // (after which stage s is no longer read and stage s+1 is complete), refills stage s's buffer
  // with stage s+NS, reads stage s+1's first fragments, then its weight slice.
  int bi = 0;                                   // stage buffer of stage s (= s mod NS)
  for (int s0 = 0; s0 < nst; s0 += UNROLL) {
#pragma unroll
    for (int d = 0; d < UNROLL; ++d) {
      const int s = s0 + d;
      if (s >= nst) break;
      const int bn = bi + 1 == NS ? 0 : bi + 1;   // stage buffer of stage s + 1
#pragma unroll
      for (int q = 0; q < kNStep; ++q) {
        const int slot = (d * kNStep + q) % kRingW;
        if (q + 1 < kNStep) {
          load_b(bq[(q + 1) & 1], bi, q + 1);
        } else {
          // this wave's share of stage s + 1 has landed and its reads of stage s are done; after
          // the barrier every wave's are, so stage s + 1 is complete and stage s's buffer is free
          __builtin_amdgcn_s_waitcnt(waitcnt_imm(kWaitStage, 0));
          asm volatile("s_barrier" ::: "memory");
          load_stage(bi, s + NS);
          load_b(bq[0], bn, 0);
        }
        load_w(ring[(slot + kRingW - 1) % kRingW], s + (q + kRingW - 1) / kNStep, (q + kRingW - 1) % kNStep);
        lgkm_wait<FT>();                        // this k-step's fragments (the next k-step's may be in flight)
        wait_w(q);                              // this k-step's weight slice
        pin(bq[q & 1]);
        pin_acc(ring[slot]);
        mma(ring[slot], bq[q & 1]);
        // keep every load in the k-step it was written in: the prefetch distances are the design
        __builtin_amdgcn_sched_barrier(0);
      }
      bi = bn;
    }
  }
  // no stage load may still be writing LDS when the tile is reused below
  __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, 0));
}

// BM_: tokens per workgroup (the configuration's own, or half of it when that fills the chip better)
// MODE: kFused contracts the whole row and finishes the tile; kSplit (split mode, grid tiles x ks)
// contracts one of ks stage ranges and stores its partial logits, and the tile's last split to
// arrive sums the tile's partials in split order and finishes the tile.
constexpr int kFused = 0, kSplit = 1;
template <bool BF16, int EPAD, int BM_, int MODE>
__global__ __launch_bounds__(kThreads, 1) void predict_kernel(Params p) {
  using Cfg = TileCfg<EPAD>;
  constexpr int WE = Cfg::WE, WT = Cfg::WT, BM = BM_;
  constexpr int EW = EPAD / WE, TW = BM / WT;
  constexpr int FE = EW / 32, FT = TW / 32;
  constexpr int NS = ring_stages(BM);
  constexpr int STAGE = BM * kStageRowBytes;     // LDS bytes of one hidden stage
  constexpr int SROW = EPAD + 4;                 // score-tile row stride in floats
  constexpr int SCORE_BYTES = BM * SROW * 4;
  constexpr int SMEM = (NS * STAGE > SCORE_BYTES) ? NS * STAGE : SCORE_BYTES;
  constexpr int LPT = EPAD / 32;                 // lanes per token in the selection phase
  constexpr int TPP = kThreads / LPT;            // token slots (lane groups) of the workgroup
  // tokens a lane group works on at once: 1 (interleaving two ran slower on MI355X)
  constexpr int NT = 1;
  constexpr int TPASS = TPP * NT;                // tokens per selection pass
  constexpr int NPASS = (BM + TPASS - 1) / TPASS;
  constexpr int GSC_TOK = TPASS < BM ? TPASS : BM;
  static_assert(WE * WT == kWaves, "every wave owns one tile slice");
  static_assert(EW % 32 == 0 && TW % 32 == 0, "wave tiles are whole 32 x 32 MFMA blocks");
  static_assert(BM % TPASS == 0 || (TPASS > BM && NT == 1 && BM % (64 / LPT) == 0),
                "every selection pass covers whole waves");

  __shared__ __attribute__((aligned(16))) char smem[SMEM];
  __shared__ int32_t hist[EPAD];
  __shared__ __attribute__((aligned(16))) float s_lbias[EPAD];   // router bias (-inf past E)
  __shared__ __attribute__((aligned(16))) float s_sbias[EPAD];   // selection bias (-inf past E)
  // selected experts per token (ids < 256), with spare slots kMaxK .. kMaxK + LPT - 1
  __shared__ int16_t sel[BM][kMaxK + LPT];
  __shared__ uint8_t kmask[BM];                 // kept lanes of each token (second phase)
  __shared__ __attribute__((aligned(16))) float grp[BM][8];   // group scores (8 groups of 32)
  __shared__ __attribute__((aligned(16))) float gsc[GSC_TOK][kMaxGroups];
  __shared__ int32_t s_flag;
  __shared__ int64_t s_red[kWaves][2];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  // wave-uniform by construction; readfirstlane keeps it (and every buffer-load offset derived
  // from it) in scalar registers
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int we = wave % WE;
  const int wt = wave / WE;
  const int tile = MODE == kSplit ? (int)(blockIdx.x / (uint32_t)p.ks) : (int)blockIdx.x;
  const int64_t row0 = (int64_t)tile * BM;
  const int E = p.E;
  constexpr int NACC = FE * FT * 16;               // accumulator registers per thread

  for (int i = tid; i < EPAD; i += kThreads) {
    hist[i] = 0;
    // padding experts get -inf in both, so their score is -inf without a per-element test
    s_lbias[i] = i < E ? (p.logit_bias ? p.logit_bias[i] : 0.f) : -__builtin_inff();
    s_sbias[i] = i < E ? (p.select_bias ? p.select_bias[i] : 0.f) : -__builtin_inff();
  }

  f32x16 acc[FE][FT];
#pragma unroll
  for (int a = 0; a < FE; ++a)
#pragma unroll
    for (int b = 0; b < FT; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

  {
    Params q = p;
    if constexpr (MODE == kSplit) {
      const int ks = (int)(blockIdx.x % (uint32_t)p.ks);
      const int chunk = (p.st_total + p.ks - 1) / p.ks;
      q.st_base = ks * chunk;
      q.nstages = p.st_total - q.st_base < chunk ? p.st_total - q.st_base : chunk;
    }
    if (row0 < p.T && q.nstages > 0)
      contract<BF16, EPAD, FE, FT, NS, BM, TW>(acc, q, row0, wave, we, wt, lane, smem);
    if constexpr (MODE == kSplit) {
      // The partial goes out with device-scope stores, which are visible to every XCD once
      // performed; each thread waits for its own, and the barrier orders them all before the
      // arrival count.  The last split to arrive reads the partials back with device-scope loads
      // (so not from a stale line of its own L2) and adds them in split order.  The loads of one
      // 16-register block go out before any of them is used, so that a tile with many registers
      // keeps them in flight together instead of waiting for each.
      float* dst = p.partial + ((size_t)blockIdx.x * NACC) * kThreads + tid;
#pragma unroll
      for (int a = 0; a < FE; ++a)
#pragma unroll
        for (int b = 0; b < FT; ++b)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            __hip_atomic_store(&dst[(size_t)((a * FT + b) * 16 + r) * kThreads], acc[a][b][r],
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, 0));
      __syncthreads();
      if (tid == 0) s_flag = atomicAdd(&p.ws_tile[tile], 1u) == (uint32_t)(p.ks - 1) ? 1 : 0;
      __syncthreads();
      if (s_flag != 1) return;
      if (tid == 0) atomicExch(&p.ws_tile[tile], 0u);   // left zeroed for the next call
      const float* src = p.partial + (size_t)tile * p.ks * NACC * kThreads + tid;
#pragma unroll
      for (int a = 0; a < FE; ++a)
#pragma unroll
        for (int b = 0; b < FT; ++b)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;
      for (int ks = 0; ks < p.ks; ++ks) {
#pragma unroll
        for (int a = 0; a < FE; ++a)
#pragma unroll
          for (int b = 0; b < FT; ++b) {
            f32x16 t;
#pragma unroll
            for (int r = 0; r < 16; ++r)
              t[r] = __hip_atomic_load(&src[((size_t)ks * NACC + (a * FT + b) * 16 + r) * kThreads],
                                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[a][b][r] += t[r];
          }
      }
    }
  }
  lds_barrier();

  // Group-limited routing where the kept groups fill exactly half of a token's lanes (as with 8
  // groups of 32 keeping 4) finishes in a second selection phase on half the lanes (compact).
  // With exactly 8 groups of 32 the group scores come straight from the score computation
  // (early): each 32-expert block of a wave is one group, split over lanes l and l + 32.
  const int ng = p.n_group;
  const int gsz = E / ng;
  const bool compact = NPASS % 2 == 0 && BM % TPASS == 0 && LPT >= 2 && ng > 1 && gsz >= 32 &&
                       p.topk_group * (gsz >> 5) * 2 == LPT;
  const bool early = compact && LPT == 8 && gsz == 32 && ng == 8 && p.kind == FB_SIGMOID &&
                     p.logit_bias == nullptr;

  // ---- logits and scores into an LDS tile S[token][expert] ------------------------
  // Lane l of a 32 x 32 block holds token (l & 31) and experts g * 8 + (l >> 5) * 4 + r in
  // register g * 4 + r.
  float* S = reinterpret_cast<float*>(smem);
  if (row0 < p.T) {
    if (p.logits) {                              // debug output of the early logits
#pragma unroll
      for (int fe = 0; fe < FE; ++fe)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int e0 = we * EW + fe * 32 + g * 8 + (lane >> 5) * 4;
#pragma unroll
          for (int ft = 0; ft < FT; ++ft) {
            const int64_t t = row0 + wt * TW + ft * 32 + (lane & 31);
            if (t < p.T) {
#pragma unroll
              for (int r = 0; r < 4; ++r)
                if (e0 + r < E) p.logits[t * E + e0 + r] = acc[fe][ft][g * 4 + r] + s_lbias[e0 + r];
            }
          }
        }
    }
    // The common case (sigmoid, no logit bias) is its own instantiation: the exponential and
    // the reciprocal dominate this phase, and it then needs only three other operations per
    // score.  A sigmoid score is never -0 (the reciprocal is positive, and +0 + -0 = +0), so only
    // the logits need the -0 -> +0 canonicalisation of the order-preserving key.
    auto emit = [&](auto sig_c, auto lbias_c, auto groups_c) {
      constexpr bool SIG = decltype(sig_c)::value, LBIAS = decltype(lbias_c)::value;
      constexpr bool GROUPS = decltype(groups_c)::value;
      // top two scores of each (expert block, token block) over this lane's 16 of its 32 experts
      float t1[FE][FT], t2[FE][FT];
#pragma unroll
      for (int fe = 0; fe < FE; ++fe)
#pragma unroll
        for (int ft = 0; ft < FT; ++ft) { t1[fe][ft] = -__builtin_inff(); t2[fe][ft] = -__builtin_inff(); }
#pragma unroll
      for (int fe = 0; fe < FE; ++fe) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int e0 = we * EW + fe * 32 + g * 8 + (lane >> 5) * 4;
          const f32x4 lb = *reinterpret_cast<const f32x4*>(s_lbias + e0);
          const f32x4 sb = *reinterpret_cast<const f32x4*>(s_sbias + e0);
#pragma unroll
          for (int ft = 0; ft < FT; ++ft) {
            const int tl = wt * TW + ft * 32 + (lane & 31);
            f32x4 sv;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const float z = LBIAS ? acc[fe][ft][g * 4 + r] + lb[r] : acc[fe][ft][g * 4 + r];
              if constexpr (SIG)
                sv[r] = __builtin_amdgcn_rcpf(1.0f + __expf(-z)) + sb[r];
              else
                sv[r] = z + 0.0f;                // -0 -> +0; padding experts stay -inf
              if constexpr (GROUPS) {
                t2[fe][ft] = __builtin_amdgcn_fmed3f(t1[fe][ft], t2[fe][ft], sv[r]);
                t1[fe][ft] = fmaxf(t1[fe][ft], sv[r]);
              }
            }
            *reinterpret_cast<f32x4*>(S + tl * SROW + e0) = sv;
          }
        }
      }
      if constexpr (GROUPS) {
        // merge with lane l + 32, which holds the block's other 16 experts of the same token: the
        // lane-half swap hands lanes 0..31 the values of lanes 32..63 (the upper half's result is
        // not used)
#pragma unroll
        for (int fe = 0; fe < FE; ++fe)
#pragma unroll
          for (int ft = 0; ft < FT; ++ft) {
            const uint32_t u1 = __float_as_uint(t1[fe][ft]), u2 = __float_as_uint(t2[fe][ft]);
            const float o1 = __uint_as_float(__builtin_amdgcn_permlane32_swap(u1, u1, false, false)[1]);
            const float o2 = __uint_as_float(__builtin_amdgcn_permlane32_swap(u2, u2, false, false)[1]);
            const float m1 = fmaxf(t1[fe][ft], o1);
            const float m2 = fmaxf(fminf(t1[fe][ft], o1), fmaxf(t2[fe][ft], o2));
            if (lane < 32)
              grp[wt * TW + ft * 32 + lane][we * FE + fe] = p.group_topn == 2 ? m1 + m2 : m1;
          }
      }
    };
    using T1 = std::integral_constant<bool, true>;
    using F0 = std::integral_constant<bool, false>;
    if (p.kind == FB_SIGMOID) {
      if (p.logit_bias) emit(T1{}, T1{}, F0{});
      else if (early) emit(T1{}, F0{}, T1{});
      else emit(T1{}, F0{}, F0{});
    } else {
      emit(F0{}, T1{}, F0{});
    }
  }
  lds_barrier();

  // ---- selection: LPT lanes per token, 32 contiguous experts per lane ------------------------
  // Lane jl reads its eight 4-expert chunks starting at chunk jl, which keeps the 16 lanes of a
  // DPP row (two tokens) on distinct LDS banks; element 4q + j of the lane is expert
  // 32 jl + 4 ((q + jl) mod 8) + j.  Tokens past T take part with no selectable expert.  With one
  // wave per SIMD nothing hides latency between waves, so each lane group works on NT tokens at
  // once as independent instruction chains.
  const int k = p.k;
  const int jl = tid % LPT;      // lane within the token group
  const int gslot = tid / LPT;   // token slot within a pass
  const int gshift = __builtin_ctz((unsigned)gsz);   // group sizes below 32 are powers of two
  auto local_of = [&](int i) { return ((((i >> 2) + jl) & 7) << 2) | (i & 3); };  // expert - 32 jl
  const int idx_base = 255 - jl * 32;        // key index bits of element i: idx_base - local_of(i)
  auto read_scores = [&](float(&dst)[32], int tlr) {
    const float* row = S + tlr * SROW + jl * 32;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(row + ((q + jl) & 7) * 4);
      dst[q * 4 + 0] = v[0]; dst[q * 4 + 1] = v[1]; dst[q * 4 + 2] = v[2]; dst[q * 4 + 3] = v[3];
    }
  };
  uint32_t idxb[32];                         // key index bits of each element
#pragma unroll
  for (int i = 0; i < 32; ++i) idxb[i] = (uint32_t)(idx_base - local_of(i));
  const RankLanes<LPT> rlanes = rank_lanes<LPT>(jl, gsz >= 32 ? gsz >> 5 : 1, E);
  // ---- finishing a token: per-lane key caches, k extraction rounds, boundary ties, histogram --
  // G lanes per token; lane jg holds 32 keys; element i of the lane is expert
  // 32 L + 4 ((i / 4 + L) mod 8) + i mod 4 (L = the lane's 32-expert slice).
  auto finish = [&](auto g_c, int jg, int tlu, bool tv, int64_t ttu, const uint32_t(&key)[32],
                    const float(&sv)[32], int L) {
    constexpr int G = decltype(g_c)::value;
    // per-lane cache of the kCache largest keys (descending), refilled by a rescan below the last
    // popped key when it runs dry
    uint32_t c[kCache];
#pragma unroll
    for (int d = 0; d < kCache; ++d) c[d] = 0;
    auto insert = [&](uint32_t v) {
#pragma unroll
      for (int d = kCache - 1; d >= 1; --d) c[d] = umed3(c[d - 1], c[d], v);
      c[0] = max(c[0], v);
    };
#pragma unroll
    for (int i = 0; i < 32; ++i) insert(key[i]);
    uint32_t last = 0xFFFFFFFFu, kth = 0, next = 0;
    // k rounds, each popping the token's largest remaining key.  Rounds are branch-free per lane:
    // the popping lane records the expert in slot r, every other lane writes its own spare slot
    // past kMaxK; a refill runs only when some lane of the wave ran dry, and lanes that did not
    // insert zeros (which leave a sorted cache unchanged).
    for (int r = 0; r < k; ++r) {
      const uint32_t h = c[0];
      const uint32_t m = group_max_u32<G>(h);
      kth = m;
      // m is never 0 here: every lane holds 32 keys and only experts >= 255 can have key 0, so
      // each of the first k <= 32 maxima is a real key with exactly one owner
      const bool mine = h == m;
      sel[tlu][mine ? r : kMaxK + jg] = (int16_t)(255 - (int)(m & 0xFFu));
#pragma unroll
      for (int d = 0; d < kCache - 1; ++d) c[d] = mine ? c[d + 1] : c[d];
      c[kCache - 1] = mine ? 0u : c[kCache - 1];
      last = mine ? m : last;
      // refill below last; a lane with nothing left below it inserts only zeros
      const bool dry = mine && c[0] == 0;
      if (__builtin_amdgcn_ballot_w64(dry) != 0) {   // rare
#pragma unroll
        for (int i = 0; i < 32; ++i) insert(dry && key[i] < last ? key[i] : 0u);
      }
    }
    // the (k+1)-th key, for the boundary test below: nothing is popped
    next = group_max_u32<G>(c[0]);
    const uint32_t tb = kth >> 8;              // score bits of the k-th key
    const bool tie = tv && (next >> 8) != 0 && (next >> 8) == tb;
    if (tie) {
      // Exact path for the boundary only.  Every key whose score bits exceed tb is selected and
      // already in place (the keys were popped in descending order); the remaining slots go to
      // the experts whose score bits equal tb, ranked by the full 64-bit key (all score bits,
      // then the inverted index), which is the exact order.
      int above = 0;
#pragma unroll
      for (int i = 0; i < 32; ++i) above += (key[i] >> 8) > tb;
#pragma unroll
      for (int off = 1; off < G; off <<= 1) above += __shfl_xor(above, off, G);
      uint64_t lastk = ~0ull;
      for (int r = above; r < k; ++r) {
        uint64_t best = 0;
#pragma unroll
        for (int i = 0; i < 32; ++i) {
          const uint32_t e = (uint32_t)(L * 32 + (((((i >> 2) + L) & 7) << 2) | (i & 3)));
          const uint64_t kk = ((uint64_t)ord_bits(sv[i] + 0.0f) << 32) | (uint64_t)(0xFFFFFFFFu - e);
          const bool ok = (key[i] >> 8) == tb && kk < lastk && kk > best;
          best = ok ? kk : best;
        }
#pragma unroll
        for (int off = 1; off < G; off <<= 1) {
          const uint64_t o = __shfl_xor(best, off, G);
          best = o > best ? o : best;
        }
        if (best == 0) break;                  // cannot happen: at least two keys share tb
        lastk = best;
        if (jg == 0) sel[tlu][r] = (int16_t)(0xFFFFFFFFu - (uint32_t)(best & 0xFFFFFFFFu));
      }
    }
    wave_lds_sync();
    if (tv) {
      for (int r = jg; r < k; r += G) {
        const int e = sel[tlu][r];
        if ((unsigned)e < (unsigned)E) atomicAdd(&hist[e], 1);
      }
    }
    if (p.topk_idx && jg == 0 && tv) {
      // debug output in exact descending score order: insertion sort of the k selected in place
      int16_t* list = sel[tlu];
      for (int r = 1; r < k; ++r) {
        const int e = list[r];
        const float se = (unsigned)e < (unsigned)E ? S[tlu * SROW + e] : -__builtin_inff();
        int q = r;
        while (q > 0) {
          const int eo = list[q - 1];
          const float so = (unsigned)eo < (unsigned)E ? S[tlu * SROW + eo] : -__builtin_inff();
          if (so > se || (so == se && eo < e)) break;
          list[q] = (int16_t)eo;
          --q;
        }
        list[q] = (int16_t)e;
      }
      for (int r = 0; r < k; ++r) p.topk_idx[ttu * k + r] = list[r];
    }
  };
  // each pass's scores are read while the previous pass is processed
  float snext[NT][32];
  if (!early) {
#pragma unroll
  for (int u = 0; u < NT; ++u)
    if (u * TPP + gslot < BM) read_scores(snext[u], u * TPP + gslot);
#pragma unroll 1
  for (int pass = 0; pass < NPASS; ++pass) {
    if (pass * TPASS + gslot >= BM) continue;  // whole waves (checked above)
    int tl[NT];
    int64_t tt[NT];
    bool tvalid[NT];
    float s[NT][32];
#pragma unroll
    for (int u = 0; u < NT; ++u) {
      tl[u] = pass * TPASS + u * TPP + gslot;
      tt[u] = row0 + tl[u];
      tvalid[u] = tt[u] < p.T;
#pragma unroll
      for (int i = 0; i < 32; ++i) s[u][i] = snext[u][i];
      if (tl[u] + TPASS < BM) read_scores(snext[u], tl[u] + TPASS);
    }
    uint32_t ob[NT][32];                       // order-preserving bits of the scores
#pragma unroll
    for (int u = 0; u < NT; ++u)
#pragma unroll
      for (int i = 0; i < 32; ++i) ob[u][i] = ord_bits(s[u][i]);
    uint32_t keep[NT];                         // bit i: element i survives the group limit
#pragma unroll
    for (int u = 0; u < NT; ++u) keep[u] = 0xFFFFFFFFu;
    if (ng > 1) {
      // group scores: sum of the group's group_topn best scores, largest first
      if (gsz >= 32) {
        // whole lanes per group: group scores and ranks stay in registers (lane exchanges inside
        // the token's LPT lanes); the else branch handles groups smaller than a lane's slice
        const int lpg = gsz >> 5;
        const bool real = jl * 32 < E;
#pragma unroll
        for (int u = 0; u < NT; ++u) {
          // top two of the lane's scores, compared as order-preserving integers (no NaN handling
          // needed: scores are finite or -inf), then merged over the group's lanes
          uint32_t k1 = 0, k2 = 0;
#pragma unroll
          for (int i = 0; i < 32; ++i) {
            k2 = umed3(k1, k2, ob[u][i]);
            k1 = max(k1, ob[u][i]);
          }
          float m1 = from_ord_bits(k1), m2 = from_ord_bits(k2);
          if (lpg > 1) top2_group(m1, m2, lpg);
          const float g = p.group_topn == 2 ? m1 + m2 : m1;
          const int rank = group_rank<LPT>(g, rlanes);
          keep[u] = (real && rank < p.topk_group) ? 0xFFFFFFFFu : 0u;
        }
      } else {
        const int gpl = 32 >> gshift;
#pragma unroll
        for (int u = 0; u < NT; ++u) {
          float* gs = gsc[u * TPP + gslot];
          for (int v = 0; v < gpl; ++v) {
            float m1 = -__builtin_inff(), m2 = -__builtin_inff();
#pragma unroll
            for (int i = 0; i < 32; ++i) {
              const bool in = (local_of(i) >> gshift) == v;
              m2 = in ? __builtin_amdgcn_fmed3f(m1, m2, s[u][i]) : m2;
              m1 = in ? fmaxf(m1, s[u][i]) : m1;
            }
            if (jl * 32 + v * gsz < E) gs[jl * gpl + v] = p.group_topn == 2 ? m1 + m2 : m1;
          }
        }
        wave_lds_sync();
#pragma unroll
        for (int u = 0; u < NT; ++u) {
          const float* gs = gsc[u * TPP + gslot];
          // rank of a group among all groups (score desc, lower index first), four scores per read
          // (rows hold kMaxGroups entries, so the reads stay in bounds)
          auto kept = [&](int g) -> bool {
            const float mine = gs[g];
            int rank = 0;
#pragma unroll 1
            for (int h4 = 0; h4 < ng; h4 += 4) {
              const f32x4 o = *reinterpret_cast<const f32x4*>(gs + h4);
#pragma unroll
              for (int j = 0; j < 4; ++j) {
                const int h = h4 + j;
                rank += (h < ng) & ((o[j] > mine) | ((o[j] == mine) & (h < g)));
              }
            }
            return rank < p.topk_group;
          };
          keep[u] = 0;
          for (int v = 0; v < gpl; ++v) {
            if (jl * 32 + v * gsz < E && kept(jl * gpl + v)) {
#pragma unroll
              for (int i = 0; i < 32; ++i) keep[u] |= (uint32_t)((local_of(i) >> gshift) == v) << i;
            }
          }
        }
      }
    }
    // 32-bit keys: the top 24 bits of the order-preserving score encoding, then 255 - expert.
    // Experts outside the kept groups (and every expert of a token past T) keep only their index
    // bits, which ranks them below every selectable expert; padding experts score -inf.
    if (compact) {
      // Only the kept groups matter from here on, and they fill exactly half of the token's lanes:
      // record which lanes they are and finish the token in the second phase below, two tokens
      // per lane group.
      const uint64_t b = __builtin_amdgcn_ballot_w64(keep[0] != 0);
      if (jl == 0) kmask[tl[0]] = (uint8_t)((b >> (lane & (64 - LPT))) & ((1u << LPT) - 1u));
      continue;
    }
    uint32_t key[32];
    if (ng == 1 || gsz >= 32) {                // the lane's experts are kept or dropped together
      const uint32_t m = tvalid[0] && keep[0] ? 0xFFFFFF00u : 0u;
#pragma unroll
      for (int i = 0; i < 32; ++i) key[i] = (ob[0][i] & m) | idxb[i];
    } else {
#pragma unroll
      for (int i = 0; i < 32; ++i) {
        const uint32_t m = tvalid[0] && ((keep[0] >> i) & 1u) ? 0xFFFFFF00u : 0u;
        key[i] = (ob[0][i] & m) | idxb[i];
      }
    }
    finish(std::integral_constant<int, LPT>{}, jl, tl[0], tvalid[0], tt[0], key, s[0], jl);
  }
  }
  if (compact) {
    // Second phase: the lane group of a token slot takes two tokens of this wave, half of its
    // lanes each; lane jb of a half reads the jb-th kept group's 32 scores back from the tile.
    constexpr int G2 = LPT / 2;
    wave_lds_sync();
    const int half = jl / G2, jb = jl % G2;
#pragma unroll 1
    for (int pb = 0; pb < NPASS / 2; ++pb) {
      const int tlc = (2 * pb + half) * TPASS + gslot;
      const int64_t ttc = row0 + tlc;
      const bool tvc = ttc < p.T;
      // the jb-th set bit of the token's kept-lane mask
      uint32_t km;
      if (early) {
        // rank groups jb and jb + 4 of the token's 8 (score desc, lower group first), then
        // gather the kept set over the half's four lanes
        const f32x4 ga = *reinterpret_cast<const f32x4*>(&grp[tlc][0]);
        const f32x4 gb = *reinterpret_cast<const f32x4*>(&grp[tlc][4]);
        const float gv[8] = {ga[0], ga[1], ga[2], ga[3], gb[0], gb[1], gb[2], gb[3]};
        uint32_t kb = 0;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int gi = jb + 4 * h;
          const float mine = h ? gv[jb + 4] : gv[jb];
          int rank = 0;
#pragma unroll
          for (int x = 0; x < 8; ++x)
            rank += (int)(gv[x] > mine) | ((int)(gv[x] == mine) & (int)(x < gi));
          kb |= (uint32_t)(rank < p.topk_group) << gi;
        }
        kb |= (uint32_t)__shfl_xor((int)kb, 1, G2);
        kb |= (uint32_t)__shfl_xor((int)kb, 2, G2);
        km = kb;
      } else {
        km = kmask[tlc];
      }
      int L = 0, seen = 0;
#pragma unroll
      for (int b = 0; b < LPT; ++b) {
        const int on = (km >> b) & 1;
        L = (on && seen == jb) ? b : L;
        seen += on;
      }
      float sc[32];
      const float* row = S + tlc * SROW + L * 32;
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(row + ((q + L) & 7) * 4);
        sc[q * 4 + 0] = v[0]; sc[q * 4 + 1] = v[1]; sc[q * 4 + 2] = v[2]; sc[q * 4 + 3] = v[3];
      }
      const uint32_t m = tvc ? 0xFFFFFF00u : 0u;
      uint32_t key[32];
#pragma unroll
      for (int i = 0; i < 32; ++i) {
        const int loc = ((((i >> 2) + L) & 7) << 2) | (i & 3);
        key[i] = (ord_bits(sc[i]) & m) | (uint32_t)(255 - (L * 32 + loc));
      }
      finish(std::integral_constant<int, G2>{}, jb, tlc, tvc, ttc, key, sc, L);
    }
  }
  lds_barrier();

  // ---- one global atomic per expert per workgroup, then the completion ticket ----------------
  // Workgroups exchange data only through device-scope atomics, which are coherent across the
  // XCDs' L2 caches without a fence.  Each thread waits for the pre-op values of its counter
  // updates (so they have been performed) before the barrier; only then does thread 0 take the
  // ticket.  The workgroup that takes the last ticket therefore reads complete counters with its
  // own atomics.  This avoids an agent-scope fence per workgroup, which on gfx950 writes back and
  // invalidates the whole L2 and serialises across the workgroups.
  int done = 0;
  for (int e = tid; e < E; e += kThreads) {
    const int v = hist[e];
    if (v) done |= atomicAdd(&p.ws_acc[e], v);
  }
  if (done < 0) s_flag = -1;                   // never true (counters stay below 2^31); uses the values
  __syncthreads();
  if (tid == 0) s_flag = (atomicAdd(p.ws_ticket, 1u) == p.nblocks - 1) ? 1 : 0;
  __syncthreads();
  if (s_flag != 1) return;

  // ---- last workgroup: counts, rank fold, max/mean; leaves the workspace zeroed -------------
  int32_t* rl = reinterpret_cast<int32_t*>(smem);
  for (int r = tid; r < p.R; r += kThreads) rl[r] = 0;
  if (tid == 0) s_flag = 0;
  __syncthreads();
  // the swap plan's tables are fetched while the counters are read, and go straight to the
  // planner's LDS (its arrays lie past the rank loads at the start of smem); R * S <= 704 and E <= 256
  static_assert(SMEM >= plan_wave_lds_bytes(wave_cap(1, 2), 1), "the planner's LDS fits");
  const PlanWaveLds pl = plan_wave_lds(smem, wave_cap(1, 2), 1);
  constexpr int kPre = (wave_cap(1, 2) + kThreads - 1) / kThreads;
  const int rs_plan = p.plan_cpl != 0 ? p.plan.R * p.plan.S : 0;
  int32_t pre[kPre];
#pragma unroll
  for (int i = 0; i < kPre; ++i) {
    const int c = tid + i * kThreads;
    pre[i] = c < rs_plan ? p.plan.slot_expert[c] : 0;
  }
  const bool pre_bytes = p.plan_cpl != 0 && p.plan.timed && tid < E;
  const int64_t preb = pre_bytes ? p.plan.expert_bytes[tid] : 0;
  for (int e = tid; e < E; e += kThreads) {
    const int v = atomicExch(&p.ws_acc[e], 0);
    p.counts[e] = v;
    if (p.plan_cpl != 0) pl.cnt[e] = v;
    const int r = p.e2r[e];
    if (r >= 0 && r < p.R) atomicAdd(&rl[r], v);
    else s_flag = 1;
  }
#pragma unroll
  for (int i = 0; i < kPre; ++i) {
    const int c = tid + i * kThreads;
    if (c < rs_plan) pl.vals[c] = pre[i];
  }
  if (pre_bytes) pl.ebytes[tid] = preb;
  __syncthreads();
  int64_t mx = 0, sum = 0;
  for (int r = tid; r < p.R; r += kThreads) {
    const int v = rl[r];
    p.rank_loads[r] = v;
    mx = v > mx ? v : mx;
    sum += v;
  }
  for (int off = 32; off > 0; off >>= 1) {
    const int64_t om = __shfl_xor(mx, off), os = __shfl_xor(sum, off);
    mx = om > mx ? om : mx;
    sum += os;
  }
  if (lane == 0) { s_red[wave][0] = mx; s_red[wave][1] = sum; }
  __syncthreads();
  if (tid == 0) {
    for (int w = 1; w < kWaves; ++w) {
      mx = s_red[w][0] > mx ? s_red[w][0] : mx;
      sum += s_red[w][1];
    }
    double ratio = sum == 0 ? 1.0 : (double)mx * (double)p.R / (double)sum;
    *p.max_mean = s_flag ? -1.0 : ratio;
    atomicExch(p.ws_ticket, 0u);
  }
  if (p.plan_cpl != 0) {
    // The swap plan of the counts just written (Alg. 1, frontier mode): the one-wave planner in
    // this workgroup's first wave, in LDS the selection no longer needs, with its tables already
    // there.  The barrier publishes every wave's entries; the other waves are done.
    __syncthreads();
    if (wave != 0) return;
    if (p.plan_cpl == 1) plan_wave_body<1, 1, true>(p.plan, pl);
    else plan_wave_body<1, 2, true>(p.plan, pl);
  }
}

__global__ void zero_kernel(uint32_t* p, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

int epad_of(int32_t E) {
  return E <= 32 ? 32 : E <= 64 ? 64 : E <= 128 ? 128 : 256;
}

// Split mode: when the tiles would occupy at most half of the CUs, the stage range of every tile
// is split over up to four workgroups (at least four stages each), so that more CUs stream the
// hidden rows and each streams a share of the router weight.
int split_count(int64_t T, int BM, int st_total, int num_cus) {
  const int64_t tiles = (T + BM - 1) / BM;
  // split mode: at most half of the CUs hold tiles, and each tile has an arrival counter
  if (T <= 0 || tiles * 2 > num_cus || tiles > kMaxSplitTiles) return 1;
  int64_t ks = num_cus / tiles;
  if (ks > 4) ks = 4;
  if (ks > st_total / 4) ks = st_total / 4;
  return ks > 1 ? (int)ks : 1;
}

// Tile height of a launch (see launch_cfg).
template <int EPAD>
int tile_rows(int64_t T, int num_cus) {
  constexpr int BM = TileCfg<EPAD>::BM;
  if (EPAD == 256) {
    const int64_t half_tiles = (T + BM / 2 - 1) / (BM / 2);
    if (T > 0 && half_tiles <= num_cus) return BM / 2;
  }
  return BM;
}

template <int EPAD>
size_t split_bytes_cfg(int64_t T, int32_t H, int32_t dtype, int num_cus) {
  const int BM = tile_rows<EPAD>(T, num_cus);
  const int st_total = (H * (dtype == FB_BF16 ? 2 : 4) + kStageRowBytes - 1) / kStageRowBytes;
  const int ks = split_count(T, BM, st_total, num_cus);
  if (ks <= 1) return 0;
  const int64_t tiles = (T + BM - 1) / BM;
  return (size_t)tiles * ks * BM * EPAD * sizeof(float);
}

template <int EPAD>
int launch_pack_cfg(const void* w, int32_t E, int32_t Hbytes, void* out, void* stream) {
  const int32_t nst = (Hbytes + kStageRowBytes - 1) / kStageRowBytes;
  const int64_t units = (int64_t)nst * EPAD * (kStageRowBytes / 16);
  const int64_t blocks64 = (units + 255) / 256;
  const int blocks = (int)(blocks64 < 4096 ? (blocks64 > 0 ? blocks64 : 1) : 4096);
  hipLaunchKernelGGL((pack_kernel<EPAD>), dim3(blocks), dim3(256), 0, static_cast<hipStream_t>(stream),
                     static_cast<const char*>(w), E, Hbytes, nst, static_cast<u32x4*>(out));
  return hipGetLastError() == hipSuccess ? FB_OK : FB_EDEVICE;
}

template <bool BF16, int EPAD, int BM>
int launch_cfg_bm(const PredictLaunch& a) {
  const int elem = BF16 ? 2 : 4;
  Params p;
  p.x = static_cast<const char*>(a.hidden);
  p.T = a.T;
  p.Hbytes = a.H * elem;
  p.ldx_bytes = (int32_t)(a.ld_hidden * elem);
  p.wpack = static_cast<const char*>(a.router_packed);
  p.E = a.E;
  p.logit_bias = a.logit_bias;
  p.select_bias = a.select_bias;
  p.kind = a.scoring.kind;
  p.k = a.scoring.k;
  p.n_group = a.scoring.n_group;
  p.topk_group = a.scoring.topk_group;
  p.group_topn = a.scoring.group_topn;
  p.e2r = a.expert_to_rank;
  p.R = a.R;
  p.counts = a.counts;
  p.rank_loads = a.rank_loads;
  p.max_mean = a.max_mean;
  p.ws_acc = reinterpret_cast<int32_t*>(static_cast<char*>(a.workspace) + kWsAccOffset);
  p.ws_ticket = reinterpret_cast<uint32_t*>(static_cast<char*>(a.workspace) + kWsTicketOffset);
  p.ws_tile = reinterpret_cast<uint32_t*>(static_cast<char*>(a.workspace) + kWsTileTicketOffset);
  p.topk_idx = a.topk_idx;
  p.logits = a.logits;
  const int64_t tiles = (a.T + BM - 1) / BM;
  p.nblocks = (uint32_t)(tiles > 0 ? tiles : 1);
  p.st_total = (p.Hbytes + kStageRowBytes - 1) / kStageRowBytes;
  p.nstages = p.st_total;
  p.st_base = 0;
  p.ks = split_count(a.T, BM, p.st_total, a.num_cus);
  p.partial = a.partial;
  p.plan_cpl = 0;
  if (a.plan != nullptr) {
    p.plan = *a.plan;
    p.plan_cpl = (int64_t)a.plan->S * a.plan->S <= 64 ? 1 : 2;
  }
  hipStream_t st = static_cast<hipStream_t>(a.stream);
  if (p.ks > 1 && a.partial != nullptr &&
      a.partial_bytes >= (size_t)tiles * p.ks * BM * EPAD * sizeof(float)) {
    hipLaunchKernelGGL((predict_kernel<BF16, EPAD, BM, kSplit>), dim3(p.nblocks * p.ks),
                       dim3(kThreads), 0, st, p);
  } else {
    p.ks = 1;
    hipLaunchKernelGGL((predict_kernel<BF16, EPAD, BM, kFused>), dim3(p.nblocks), dim3(kThreads),
                       0, st, p);
  }
  return hipGetLastError() == hipSuccess ? FB_OK : FB_EDEVICE;
}

template <bool BF16, int EPAD>
int launch_cfg(const PredictLaunch& a) {
  constexpr int BM = TileCfg<EPAD>::BM;
  // Half-height tiles when the full-height grid would leave CUs idle and the half-height one still
  // fits in a single wave of workgroups: every CU then streams the weight for fewer tokens.
  if constexpr (EPAD == 256) {
    if (tile_rows<EPAD>(a.T, a.num_cus) == BM / 2) return launch_cfg_bm<BF16, EPAD, BM / 2>(a);
  }
  return launch_cfg_bm<BF16, EPAD, BM>(a);
}

template <bool BF16>
int launch_dtype(const PredictLaunch& a) {
  switch (epad_of(a.E)) {
    case 32: return launch_cfg<BF16, 32>(a);
    case 64: return launch_cfg<BF16, 64>(a);
    case 128: return launch_cfg<BF16, 128>(a);
    default: return launch_cfg<BF16, 256>(a);
  }
}

}  // namespace

size_t router_packed_bytes(int32_t E, int32_t H, int32_t dtype) {
  const int64_t Hbytes = (int64_t)H * (dtype == FB_BF16 ? 2 : 4);
  const int64_t nst = (Hbytes + kStageRowBytes - 1) / kStageRowBytes;
  return (size_t)(nst * epad_of(E) * kStageRowBytes);
}

int launch_pack(const void* router_w, int32_t E, int32_t H, int32_t dtype, void* packed, void* stream) {
  (void)hipGetLastError();
  const int32_t Hbytes = H * (dtype == FB_BF16 ? 2 : 4);
  switch (epad_of(E)) {
    case 32: return launch_pack_cfg<32>(router_w, E, Hbytes, packed, stream);
    case 64: return launch_pack_cfg<64>(router_w, E, Hbytes, packed, stream);
    case 128: return launch_pack_cfg<128>(router_w, E, Hbytes, packed, stream);
    default: return launch_pack_cfg<256>(router_w, E, Hbytes, packed, stream);
  }
}

size_t split_workspace_bytes(int64_t T, int32_t E, int32_t H, int32_t dtype, int num_cus) {
  switch (epad_of(E)) {
    case 32: return split_bytes_cfg<32>(T, H, dtype, num_cus);
    case 64: return split_bytes_cfg<64>(T, H, dtype, num_cus);
    case 128: return split_bytes_cfg<128>(T, H, dtype, num_cus);
    default: return split_bytes_cfg<256>(T, H, dtype, num_cus);
  }
}

int launch_predict(const PredictLaunch& a) {
  (void)hipGetLastError();
  return a.dtype == FB_BF16 ? launch_dtype<true>(a) : launch_dtype<false>(a);
}

int launch_workspace_zero(void* workspace, size_t bytes, void* stream) {
  (void)hipGetLastError();
  hipLaunchKernelGGL(zero_kernel, dim3(1), dim3(256), 0, static_cast<hipStream_t>(stream),
                     static_cast<uint32_t*>(workspace), bytes / 4);
  return hipGetLastError() == hipSuccess ? FB_OK : FB_EDEVICE;
}

// ---- scratch of the no-allocation entry point ----------------------------------------------------
// fb_predict_load_packed_noalloc runs the kernels above with this array as its workspace.  In host
// code its name is not a device address: the address of each device's copy comes from
// hipGetSymbolAddress and is kept per device.
static __device__ __align__(256) char scratch[kNoAllocScratchBytes];

namespace {
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxScratchDevices];
}  // namespace

int noalloc_scratch(void** ptr, void* stream) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) {
    (void)hipGetLastError();
    return FB_EDEVICE;
  }
  if (dev >= kMaxScratchDevices) return FB_EUNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_addr[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) {
      (void)hipGetLastError();
      return FB_EDEVICE;
    }
    // The header (accumulators and ticket) must start at zero; every completed call leaves it
    // zeroed again.  A fill kernel rather than a memset node, so a first call made under graph
    // capture stays valid on every replay.
    const int zc = launch_workspace_zero(p, kWsBytes, stream);
    if (zc != FB_OK) return zc;
    g_scratch_addr[dev] = p;
  }
  *ptr = g_scratch_addr[dev];
  return FB_OK;
}

}  // namespace fb
