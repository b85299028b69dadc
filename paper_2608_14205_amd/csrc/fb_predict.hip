// Fused residual workload predictor for gfx950 (MI355X).
//
// One kernel computes, for a tile of tokens, the early router logits (Sec. "Residual Workload
// Prediction", Eq. 2 with the linear router of Eq. 4), the routed model's scores and its
// (optionally group-limited) top-k selection, and the per-expert token histogram of Eq. 5.  The
// last workgroup to finish folds the histogram into per-rank loads under the expert-to-rank
// placement (Alg. 1, second step) and computes the max-to-mean ratio (Sec. "Metrics").
//
// Data flow of one workgroup (4 waves, 256 threads, one workgroup per CU):
//   * hidden rows stream from HBM through raw buffer loads (bounds-checked: rows past T read as
//     zero) into registers, kDepth stages ahead, then into a double-buffered LDS stage that all
//     waves share;
//   * each wave owns a slice of the experts; its router-weight fragments come straight from L2
//     into registers (same prefetch distance, so the in-order vmcnt waits never stall on a later
//     hidden stage);
//   * v_mfma_f32_16x16x32_bf16 (or 16x16x4 f32) with the router weight as the A operand
//     (M = experts) and the hidden tile as B (N = tokens), so each lane ends with four consecutive
//     experts of one token;
//   * the logits never leave the chip: scores go to an LDS tile, EPAD/16 lanes cooperate on one
//     token, and the histogram is privatised in LDS with one global atomic per expert per
//     workgroup.
//
// Selection is exact in float32 with ties to the lower expert index.  The fast path ranks 32-bit
// keys (top 24 bits of the order-preserving score encoding, then 255 - expert); its set equals the
// exact top-k whenever the k-th and (k+1)-th keys differ in their score bits, and tokens where they
// do not take an exact 64-bit path.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fb_internal.h"

namespace fb {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kSlabBytes = 64;                  // bytes of a row feeding one MFMA k-slab
constexpr int kNSlab = 2;                       // k-slabs per pipeline stage
constexpr int kStageRowBytes = kSlabBytes * kNSlab;
constexpr int kDepth = 3;                       // pipeline stages in flight
constexpr int kChunk = 1024;                    // one (slab, 16-token fragment): 64 lanes x 16 B
constexpr int kMaxK = FB_MAX_TOPK;
constexpr int kMaxGroups = 32;
constexpr uint32_t kRsrcWord3 = 0x00020000u;    // raw buffer, 32-bit dwords

// Tile shapes: WE waves along experts x WT waves along tokens, BM tokens per workgroup.
template <int EPAD> struct TileCfg;
template <> struct TileCfg<256> { static constexpr int WE = 4, WT = 1, BM = 128; };
template <> struct TileCfg<128> { static constexpr int WE = 4, WT = 1, BM = 64; };
template <> struct TileCfg<64> { static constexpr int WE = 4, WT = 1, BM = 64; };
template <> struct TileCfg<32> { static constexpr int WE = 2, WT = 2, BM = 64; };
template <> struct TileCfg<16> { static constexpr int WE = 1, WT = 4, BM = 64; };

struct Params {
  const char* x;
  int64_t T;
  int32_t Hbytes;
  int32_t ldx_bytes;
  const char* w;
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
  int32_t* topk_idx;
  float* logits;
  uint32_t nblocks;
  int32_t nstages;
  int32_t tail_half;
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

// Order-preserving map of float bits to unsigned (for finite values; -0 is canonicalised first).
__device__ __forceinline__ uint32_t ord_bits(float s) {
  uint32_t u = __float_as_uint(s);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
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

template <bool BF16, int EPAD>
__global__ __launch_bounds__(kThreads, 1) void predict_kernel(Params p) {
  using Cfg = TileCfg<EPAD>;
  constexpr int WE = Cfg::WE, WT = Cfg::WT, BM = Cfg::BM;
  constexpr int EW = EPAD / WE, TW = BM / WT;
  constexpr int FE = EW / 16, FT = TW / 16, NF = BM / 16;
  constexpr int CPW = kNSlab * NF / 4;           // hidden chunks each wave loads per stage
  constexpr int STAGE_BYTES = kNSlab * NF * kChunk;
  constexpr int SROW = EPAD + 4;                 // score-tile row stride in floats
  constexpr int SCORE_BYTES = BM * SROW * 4;
  constexpr int SMEM = (2 * STAGE_BYTES > SCORE_BYTES) ? 2 * STAGE_BYTES : SCORE_BYTES;
  constexpr int LPT = EPAD / 16;                 // lanes per token in the selection phase
  constexpr int TPP = kThreads / LPT;            // tokens per selection pass
  constexpr int NPASS = (BM + TPP - 1) / TPP;
  constexpr int GSC_TOK = TPP < BM ? TPP : BM;
  static_assert(CPW >= 1 && (kNSlab * NF) % 4 == 0, "stage must split over 4 waves");

  __shared__ __attribute__((aligned(16))) char smem[SMEM];
  __shared__ int32_t hist[EPAD];
  __shared__ int32_t sel[BM][kMaxK + 1];
  __shared__ float gsc[GSC_TOK][kMaxGroups];
  __shared__ int32_t s_flag;
  __shared__ int64_t s_red[kThreads / 64][2];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int we = wave % WE;
  const int wt = wave / WE;
  const int64_t row0 = (int64_t)blockIdx.x * BM;
  const int E = p.E;

  for (int i = tid; i < EPAD; i += kThreads) hist[i] = 0;

  f32x4 acc[FE][FT];
#pragma unroll
  for (int a = 0; a < FE; ++a)
#pragma unroll
    for (int b = 0; b < FT; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (row0 < p.T) {
    // ---- router GEMM: acc[e][t] = sum_h W[e,h] * X[t,h] -------------------------------------
    const int64_t rows = (p.T - row0) < BM ? (p.T - row0) : BM;
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(p.x + row0 * (int64_t)p.ldx_bytes), (short)0, (int)(rows * p.ldx_bytes), kRsrcWord3);
    const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
        (void*)p.w, (short)0, E * p.Hbytes, kRsrcWord3);

    uint32_t xoff[CPW];
#pragma unroll
    for (int i = 0; i < CPW; ++i) {
      const int c = wave * CPW + i, s = c / NF, f = c % NF;
      xoff[i] = (uint32_t)((f * 16 + (lane & 15)) * p.ldx_bytes + s * kSlabBytes + (lane >> 4) * 16);
    }
    uint32_t woff[FE];
#pragma unroll
    for (int fe = 0; fe < FE; ++fe) {
      const int erow = we * EW + fe * 16 + (lane & 15);
      woff[fe] = (uint32_t)(erow * p.Hbytes + (lane >> 4) * 16);
    }

    u32x4 xa[kDepth][CPW];
    u32x4 wa[kDepth][FE][kNSlab];
    const int nst = p.nstages;
    // A slab whose k-range starts at or past H (the padded stages of the last unrolled round and
    // the second slab of a half-width last stage) is loaded with the top bit set in the per-lane
    // offset: the hardware range check (which covers the per-lane offset) fails, the load returns
    // zeros and no memory is touched.  Every load is then unconditional, which keeps the
    // compiler's in-order vmcnt accounting exact (a conditional load would force it to assume the
    // loop's later loads might be missing and to wait for everything).
    const int nst_pad = ((nst + kDepth - 1) / kDepth) * kDepth;
    auto slab_ok = [&](int st, int s) -> bool { return st * kStageRowBytes + s * kSlabBytes < p.Hbytes; };

#define FB_LOAD_X(D, ST)                                                                        \
  {                                                                                             \
    const int st_ = (ST);                                                                       \
    _Pragma("unroll") for (int i = 0; i < CPW; ++i) {                                           \
      const int s_ = (wave * CPW + i) / NF;                                                     \
      const bool ok_ = slab_ok(st_, s_);                                                        \
      xa[D][i] = __builtin_amdgcn_raw_buffer_load_b128(xr, xoff[i] | (ok_ ? 0u : 0x80000000u),  \
                                                       ok_ ? st_ * kStageRowBytes : 0, 2);      \
    }                                                                                           \
  }
#define FB_LOAD_W(D, ST)                                                                        \
  {                                                                                             \
    const int st_ = (ST);                                                                       \
    _Pragma("unroll") for (int s = 0; s < kNSlab; ++s) {                                        \
      const bool ok_ = slab_ok(st_, s);                                                         \
      _Pragma("unroll") for (int fe = 0; fe < FE; ++fe) wa[D][fe][s] =                          \
          __builtin_amdgcn_raw_buffer_load_b128(                                                \
              wr, (woff[fe] + s * kSlabBytes) | (ok_ ? 0u : 0x80000000u),                       \
              ok_ ? st_ * kStageRowBytes : 0, 0);                                               \
    }                                                                                           \
  }

    // Issue order X(0), W(0), X(1), W(1), ... matches the steady state below, so the wait counts
    // the compiler derives at the loop header are exact.
#pragma unroll
    for (int d = 0; d < kDepth; ++d) {
      FB_LOAD_X(d, d)
      __builtin_amdgcn_sched_barrier(0);
      FB_LOAD_W(d, d)
      __builtin_amdgcn_sched_barrier(0);
    }

    for (int st0 = 0; st0 < nst_pad; st0 += kDepth) {
#pragma unroll
      for (int d = 0; d < kDepth; ++d) {
        const int st = st0 + d;
        char* buf = smem + (st & 1) * STAGE_BYTES;
#pragma unroll
        for (int i = 0; i < CPW; ++i)
          *reinterpret_cast<u32x4*>(buf + (wave * CPW + i) * kChunk + lane * 16) = xa[d][i];
        FB_LOAD_X(d, st + kDepth)
        __builtin_amdgcn_sched_barrier(0);
        lds_barrier();
        // the second slab of a half-width last stage lies past H: skip it (padded stages are zero)
        const bool half = (st == nst - 1) && p.tail_half;
        u32x4 bfr[kNSlab][FT];
#pragma unroll
        for (int ft = 0; ft < FT; ++ft)
          bfr[0][ft] = *reinterpret_cast<const u32x4*>(buf + (wt * FT + ft) * kChunk + lane * 16);
#pragma unroll
        for (int s = 0; s < kNSlab; ++s) {
          if (s + 1 < kNSlab) {
#pragma unroll
            for (int ft = 0; ft < FT; ++ft)
              bfr[s + 1][ft] = *reinterpret_cast<const u32x4*>(
                  buf + ((s + 1) * NF + wt * FT + ft) * kChunk + lane * 16);
          }
          if (s == 0 || !half) {
#pragma unroll
            for (int fe = 0; fe < FE; ++fe) {
#pragma unroll
              for (int ft = 0; ft < FT; ++ft) {
                if constexpr (BF16) {
                  acc[fe][ft] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                      __builtin_bit_cast(bf16x8, wa[d][fe][s]), __builtin_bit_cast(bf16x8, bfr[s][ft]),
                      acc[fe][ft], 0, 0, 0);
                } else {
                  const f32x4 av = __builtin_bit_cast(f32x4, wa[d][fe][s]);
                  const f32x4 bv = __builtin_bit_cast(f32x4, bfr[s][ft]);
#pragma unroll
                  for (int q = 0; q < 4; ++q)
                    acc[fe][ft] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[q], bv[q], acc[fe][ft], 0, 0, 0);
                }
              }
            }
          }
        }
        __builtin_amdgcn_sched_barrier(0);
        FB_LOAD_W(d, st + kDepth)
        __builtin_amdgcn_sched_barrier(0);
      }
    }
#undef FB_LOAD_X
#undef FB_LOAD_W
  }
  lds_barrier();

  // ---- scores into an LDS tile S[token][expert] ------------------------------------------------
  float* S = reinterpret_cast<float*>(smem);
  if (row0 < p.T) {
#pragma unroll
    for (int fe = 0; fe < FE; ++fe) {
      const int e0 = we * EW + fe * 16 + (lane >> 4) * 4;
      float lb[4], sb[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int e = e0 + r;
        lb[r] = (p.logit_bias && e < E) ? p.logit_bias[e] : 0.f;
        sb[r] = (p.select_bias && e < E) ? p.select_bias[e] : 0.f;
      }
#pragma unroll
      for (int ft = 0; ft < FT; ++ft) {
        const int tl = wt * TW + ft * 16 + (lane & 15);
        const int64_t t = row0 + tl;
        f32x4 sv;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int e = e0 + r;
          const float z = acc[fe][ft][r] + lb[r];
          if (p.logits && t < p.T && e < E) p.logits[t * E + e] = z;
          float s;
          if (p.kind == FB_SIGMOID) {
            s = __builtin_amdgcn_rcpf(1.0f + __expf(-z)) + sb[r];
          } else {
            s = z;
          }
          sv[r] = (e < E) ? s + 0.0f : -__builtin_inff();
        }
        *reinterpret_cast<f32x4*>(S + tl * SROW + e0) = sv;
      }
    }
  }
  lds_barrier();

  // ---- selection: LPT lanes per token, 16 contiguous experts per lane ------------------------
  const int k = p.k;
  const int jl = tid % LPT;      // lane within the token group
  const int gslot = tid / LPT;   // token slot within a pass
#pragma unroll 1
  for (int pass = 0; pass < NPASS; ++pass) {
    const int tl = pass * TPP + gslot;
    if (tl >= BM) continue;                    // uniform per token group
    const int64_t t = row0 + tl;
    if (t >= p.T) continue;                    // uniform per token group

    float s[16];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(S + tl * SROW + jl * 16 + q * 4);
      s[q * 4 + 0] = v[0]; s[q * 4 + 1] = v[1]; s[q * 4 + 2] = v[2]; s[q * 4 + 3] = v[3];
    }
    uint32_t keep = 0xFFFFu;                   // bit i: expert jl*16+i survives the group limit
    if (p.n_group > 1) {
      const int gsz = E / p.n_group;
      float* gs = gsc[gslot];
      if (gsz >= 16) {
        const int lpg = gsz >> 4;
        float m1 = -__builtin_inff(), m2 = -__builtin_inff();
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float v = s[i];
          m2 = __builtin_amdgcn_fmed3f(m1, m2, v);
          m1 = fmaxf(m1, v);
        }
        top2_group(m1, m2, lpg);
        const int g = (jl * 16) / gsz;
        const float score = p.group_topn == 2 ? m1 + m2 : m1;
        if ((jl & (lpg - 1)) == 0 && jl * 16 < E) gs[g] = score;
      } else {
        const int gpl = 16 / gsz;
        for (int u = 0; u < gpl; ++u) {
          float m1 = -__builtin_inff(), m2 = -__builtin_inff();
          for (int i = u * gsz; i < (u + 1) * gsz; ++i) {
            const float v = s[i];
            m2 = __builtin_amdgcn_fmed3f(m1, m2, v);
            m1 = fmaxf(m1, v);
          }
          const int g = jl * gpl + u;
          if (jl * 16 + u * gsz < E) gs[g] = p.group_topn == 2 ? m1 + m2 : m1;
        }
      }
      wave_lds_sync();
      keep = 0;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int e = jl * 16 + i;
        if (e < E) {
          const int g = e / gsz;
          const float mine = gs[g];
          int rank = 0;
          for (int h = 0; h < p.n_group; ++h) {
            const float o = gs[h];
            rank += (o > mine) || (o == mine && h < g);
          }
          if (rank < p.topk_group) keep |= 1u << i;
        }
      }
    }

    uint32_t key[16];
    int nvalid = 0;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int e = jl * 16 + i;
      const bool valid = (e < E) && ((keep >> i) & 1u);
      key[i] = valid ? ((ord_bits(s[i]) & 0xFFFFFF00u) | (uint32_t)(255 - e)) : 0u;
      nvalid += valid;
    }
    uint32_t t1 = 0, t2 = 0, t3 = 0;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const uint32_t v = key[i];
      const uint32_t n3 = umed3(t2, t3, v);
      const uint32_t n2 = umed3(t1, t2, v);
      t1 = max(t1, v); t2 = n2; t3 = n3;
    }
    int npop = 0;
    uint32_t last = 0xFFFFFFFFu, kth = 0, next = 0;
    const int rounds = k + 1;
    for (int r = 0; r < rounds; ++r) {
      const uint32_t h = t1;
      const uint32_t m = group_max_u32<LPT>(h);
      if (r == k - 1) kth = m;
      if (r == k) next = m;
      if (m != 0 && h == m) {
        if (r < k) sel[tl][r] = 255 - (int)(m & 0xFFu);
        t1 = t2; t2 = t3; t3 = 0; ++npop; last = m;
        if (t1 == 0 && npop < nvalid) {        // this lane's cached top-3 ran dry: rescan below `last`
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const uint32_t v = key[i] < last ? key[i] : 0u;
            const uint32_t n3 = umed3(t2, t3, v);
            const uint32_t n2 = umed3(t1, t2, v);
            t1 = max(t1, v); t2 = n2; t3 = n3;
          }
        }
      }
    }
    const bool tie = next != 0 && (next >> 8) == (kth >> 8);
    if (tie) {
      // exact path: 64-bit keys (full order-preserving score bits, then the inverted index)
      uint64_t lastk = ~0ull;
      for (int r = 0; r < k; ++r) {
        uint64_t best = 0;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int e = jl * 16 + i;
          const uint64_t kk = ((uint64_t)ord_bits(s[i]) << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)e);
          const bool ok = key[i] != 0 && kk < lastk && kk > best;
          best = ok ? kk : best;
        }
#pragma unroll
        for (int off = 1; off < LPT; off <<= 1) {
          const uint64_t o = __shfl_xor(best, off, LPT);
          best = o > best ? o : best;
        }
        if (best == 0) break;                  // cannot happen with >= k selectable experts
        lastk = best;
        if (jl == 0) sel[tl][r] = (int)(0xFFFFFFFFu - (uint32_t)(best & 0xFFFFFFFFu));
      }
    }
    wave_lds_sync();
    for (int r = jl; r < k; r += LPT) {
      const int e = sel[tl][r];
      if ((unsigned)e < (unsigned)E) atomicAdd(&hist[e], 1);
    }
    if (p.topk_idx && jl == 0) {
      // debug output in exact descending score order: insertion sort of the k selected in place
      int* list = sel[tl];
      for (int r = 1; r < k; ++r) {
        const int e = list[r];
        const float se = (unsigned)e < (unsigned)E ? S[tl * SROW + e] : -__builtin_inff();
        int q = r;
        while (q > 0) {
          const int eo = list[q - 1];
          const float so = (unsigned)eo < (unsigned)E ? S[tl * SROW + eo] : -__builtin_inff();
          if (so > se || (so == se && eo < e)) break;
          list[q] = eo;
          --q;
        }
        list[q] = e;
      }
      for (int r = 0; r < k; ++r) p.topk_idx[t * k + r] = list[r];
    }
  }
  lds_barrier();

  // ---- one global atomic per expert per workgroup, then the completion ticket ----------------
  for (int e = tid; e < E; e += kThreads) {
    const int v = hist[e];
    if (v) atomicAdd(&p.ws_acc[e], v);
  }
  __threadfence();
  __syncthreads();
  if (tid == 0) s_flag = (atomicAdd(p.ws_ticket, 1u) == p.nblocks - 1) ? 1 : 0;
  __syncthreads();
  if (!s_flag) return;
  __threadfence();

  // ---- last workgroup: counts, rank fold, max/mean; leaves the workspace zeroed -------------
  int32_t* rl = reinterpret_cast<int32_t*>(smem);
  for (int r = tid; r < p.R; r += kThreads) rl[r] = 0;
  if (tid == 0) s_flag = 0;
  __syncthreads();
  for (int e = tid; e < E; e += kThreads) {
    const int v = atomicExch(&p.ws_acc[e], 0);
    p.counts[e] = v;
    const int r = p.e2r[e];
    if (r >= 0 && r < p.R) atomicAdd(&rl[r], v);
    else s_flag = 1;
  }
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
    for (int w = 1; w < kThreads / 64; ++w) {
      mx = s_red[w][0] > mx ? s_red[w][0] : mx;
      sum += s_red[w][1];
    }
    double ratio = sum == 0 ? 1.0 : (double)mx * (double)p.R / (double)sum;
    *p.max_mean = s_flag ? -1.0 : ratio;
    atomicExch(p.ws_ticket, 0u);
  }
}

__global__ void zero_kernel(uint32_t* p, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

template <bool BF16, int EPAD>
int launch_cfg(const PredictLaunch& a) {
  using Cfg = TileCfg<EPAD>;
  const int elem = BF16 ? 2 : 4;
  Params p;
  p.x = static_cast<const char*>(a.hidden);
  p.T = a.T;
  p.Hbytes = a.H * elem;
  p.ldx_bytes = (int32_t)(a.ld_hidden * elem);
  p.w = static_cast<const char*>(a.router_w);
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
  p.topk_idx = a.topk_idx;
  p.logits = a.logits;
  const int64_t tiles = (a.T + Cfg::BM - 1) / Cfg::BM;
  p.nblocks = (uint32_t)(tiles > 0 ? tiles : 1);
  p.nstages = (p.Hbytes + kStageRowBytes - 1) / kStageRowBytes;
  p.tail_half = (p.Hbytes % kStageRowBytes) != 0;
  hipLaunchKernelGGL((predict_kernel<BF16, EPAD>), dim3(p.nblocks), dim3(kThreads), 0,
                     static_cast<hipStream_t>(a.stream), p);
  return hipGetLastError() == hipSuccess ? FB_OK : FB_EDEVICE;
}

template <bool BF16>
int launch_dtype(const PredictLaunch& a) {
  if (a.E <= 16) return launch_cfg<BF16, 16>(a);
  if (a.E <= 32) return launch_cfg<BF16, 32>(a);
  if (a.E <= 64) return launch_cfg<BF16, 64>(a);
  if (a.E <= 128) return launch_cfg<BF16, 128>(a);
  return launch_cfg<BF16, 256>(a);
}

}  // namespace

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

}  // namespace fb
