// Prediction-quality diagnostics on the device (Sec. "Metrics" and the prediction-quality study):
// the top-k hit rate of the early pass against the actual routing, the mean per-token cosine
// similarity of two row-major matrices (hidden states h_{l-1} vs H_l, or early vs actual logits),
// and the fold of a count vector into rank loads under a placement (the realised balance of the
// actual routing under the old or the planned placement).
//
// Everything is deterministic: hits are an integer sum; cosines are summed per wave in a fixed
// order into a workspace and reduced by one workgroup in index order.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fb_internal.h"

namespace fb {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kQThreads = 256;
constexpr int kQWaves = kQThreads / 64;

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

// One token per thread: the predicted experts become a bit set, the actual ones are looked up.
__global__ __launch_bounds__(kQThreads) void hits_kernel(const int32_t* __restrict__ pred,
                                                         const int32_t* __restrict__ act, int64_t T,
                                                         int32_t k, unsigned long long* __restrict__ hits) {
  __shared__ unsigned long long s_part[kQWaves];
  const int64_t t = blockIdx.x * (int64_t)kQThreads + threadIdx.x;
  unsigned long long h = 0;
  if (t < T) {
    uint32_t bits[FB_MAX_EXPERTS / 32];
#pragma unroll
    for (int w = 0; w < FB_MAX_EXPERTS / 32; ++w) bits[w] = 0;
    for (int j = 0; j < k; ++j) {
      const uint32_t e = (uint32_t)pred[t * k + j];
      if (e < FB_MAX_EXPERTS) {
#pragma unroll
        for (int w = 0; w < FB_MAX_EXPERTS / 32; ++w) bits[w] |= (w == (int)(e >> 5)) ? 1u << (e & 31) : 0u;
      }
    }
    for (int j = 0; j < k; ++j) {
      const uint32_t e = (uint32_t)act[t * k + j];
      uint32_t word = 0;
#pragma unroll
      for (int w = 0; w < FB_MAX_EXPERTS / 32; ++w) word = (w == (int)(e >> 5)) ? bits[w] : word;
      h += (e < FB_MAX_EXPERTS) && ((word >> (e & 31)) & 1u);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) h += __shfl_xor(h, off);
  if ((threadIdx.x & 63) == 0) s_part[threadIdx.x >> 6] = h;
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long sum = 0;
    for (int w = 0; w < kQWaves; ++w) sum += s_part[w];
    if (sum) atomicAdd(hits, sum);
  }
}

__global__ void zero_u64_kernel(unsigned long long* p) { *p = 0ull; }

// hit rate = hits / (T * k), 1.0 for an empty batch
__global__ void rate_kernel(const unsigned long long* hits, int64_t slots, double* rate) {
  *rate = slots > 0 ? (double)*hits / (double)slots : 1.0;
}

// One wave per row at a time; 16-byte loads; products and sums in double.  Each wave writes the sum
// of the cosines of the rows it handled to partial[wave id].
template <bool BF16>
__global__ __launch_bounds__(kQThreads) void cosine_kernel(const char* __restrict__ a,
                                                           const char* __restrict__ b, int64_t rows,
                                                           int32_t cols, int64_t lda_bytes,
                                                           int64_t ldb_bytes, double* __restrict__ partial) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * kQWaves + (threadIdx.x >> 6);
  const int64_t nwaves = (int64_t)gridDim.x * kQWaves;
  constexpr int kPer = BF16 ? 8 : 4;          // elements per 16-byte chunk
  const int chunks = cols / kPer;
  double acc = 0.0;
  for (int64_t r = wave; r < rows; r += nwaves) {
    const u32x4* ra = reinterpret_cast<const u32x4*>(a + r * lda_bytes);
    const u32x4* rb = reinterpret_cast<const u32x4*>(b + r * ldb_bytes);
    double dot = 0.0, aa = 0.0, bb = 0.0;
    for (int c = lane; c < chunks; c += 64) {
      const u32x4 va = __builtin_nontemporal_load(ra + c);
      const u32x4 vb = __builtin_nontemporal_load(rb + c);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if constexpr (BF16) {
          const double x0 = (double)__uint_as_float(va[q] << 16), x1 = (double)__uint_as_float(va[q] & 0xFFFF0000u);
          const double y0 = (double)__uint_as_float(vb[q] << 16), y1 = (double)__uint_as_float(vb[q] & 0xFFFF0000u);
          dot = fma(x0, y0, dot); dot = fma(x1, y1, dot);
          aa = fma(x0, x0, aa); aa = fma(x1, x1, aa);
          bb = fma(y0, y0, bb); bb = fma(y1, y1, bb);
        } else {
          const double x = (double)__uint_as_float(va[q]), y = (double)__uint_as_float(vb[q]);
          dot = fma(x, y, dot); aa = fma(x, x, aa); bb = fma(y, y, bb);
        }
      }
    }
    dot = wave_sum_f64(dot);
    aa = wave_sum_f64(aa);
    bb = wave_sum_f64(bb);
    acc += dot / (sqrt(aa) * sqrt(bb));
  }
  if (lane == 0) partial[wave] = acc;
}

// Sum of the per-wave partials in index order (one workgroup), divided by the row count.
__global__ __launch_bounds__(kQThreads) void mean_kernel(const double* __restrict__ partial, int64_t n,
                                                         int64_t rows, double* __restrict__ out) {
  __shared__ double s[kQThreads];
  double v = 0.0;
  const int64_t per = (n + kQThreads - 1) / kQThreads;   // contiguous slice per thread
  for (int64_t i = threadIdx.x * per; i < n && i < (threadIdx.x + 1) * per; ++i) v += partial[i];
  s[threadIdx.x] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    double sum = 0.0;
    for (int i = 0; i < kQThreads; ++i) sum += s[i];
    *out = rows > 0 ? sum / (double)rows : 1.0;
  }
}

// Rank loads and max-to-mean of a count vector under a placement (one workgroup).
__global__ __launch_bounds__(kQThreads) void fold_kernel(const int32_t* __restrict__ counts, int32_t E,
                                                         const int32_t* __restrict__ e2r, int32_t R,
                                                         int32_t* __restrict__ rank_loads,
                                                         double* __restrict__ max_mean) {
  __shared__ int32_t rl[FB_MAX_RANKS];
  __shared__ int32_t s_bad;
  __shared__ long long s_mx[kQWaves], s_sum[kQWaves];
  const int tid = threadIdx.x;
  if (tid == 0) s_bad = 0;
  for (int r = tid; r < R; r += kQThreads) rl[r] = 0;
  __syncthreads();
  for (int e = tid; e < E; e += kQThreads) {
    const int r = e2r[e];
    if (r >= 0 && r < R) atomicAdd(&rl[r], counts[e]);
    else s_bad = 1;
  }
  __syncthreads();
  long long mx = 0, sum = 0;
  for (int r = tid; r < R; r += kQThreads) {
    const int v = rl[r];
    rank_loads[r] = v;
    mx = v > mx ? v : mx;
    sum += v;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const long long om = __shfl_xor(mx, off), os = __shfl_xor(sum, off);
    mx = om > mx ? om : mx;
    sum += os;
  }
  if ((tid & 63) == 0) { s_mx[tid >> 6] = mx; s_sum[tid >> 6] = sum; }
  __syncthreads();
  if (tid == 0) {
    for (int w = 1; w < kQWaves; ++w) { mx = s_mx[w] > mx ? s_mx[w] : mx; sum += s_sum[w]; }
    *max_mean = s_bad ? -1.0 : (sum == 0 ? 1.0 : (double)mx * (double)R / (double)sum);
  }
}

}  // namespace

size_t cosine_workspace_bytes() { return (size_t)kCosineBlocks * kQWaves * sizeof(double); }

int launch_hits(const int32_t* pred, const int32_t* act, int64_t T, int32_t k, int64_t* hits,
                double* rate, void* stream) {
  (void)hipGetLastError();
  hipStream_t st = static_cast<hipStream_t>(stream);
  auto* h = reinterpret_cast<unsigned long long*>(hits);
  hipLaunchKernelGGL(zero_u64_kernel, dim3(1), dim3(1), 0, st, h);
  if (T > 0) {
    const int64_t blocks = (T + kQThreads - 1) / kQThreads;
    hipLaunchKernelGGL(hits_kernel, dim3((unsigned)blocks), dim3(kQThreads), 0, st, pred, act, T, k, h);
  }
  if (rate) hipLaunchKernelGGL(rate_kernel, dim3(1), dim3(1), 0, st, h, T * (int64_t)k, rate);
  return hipGetLastError() == hipSuccess ? FB_OK : FB_EDEVICE;
}

int launch_cosine(const void* a, const void* b, int64_t rows, int32_t cols, int64_t lda, int64_t ldb,
                  int32_t dtype, double* out, void* workspace, void* stream) {
  (void)hipGetLastError();
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int elem = dtype == FB_BF16 ? 2 : 4;
  double* partial = static_cast<double*>(workspace);
  const int64_t waves_needed = rows;
  const int64_t blocks64 = (waves_needed + kQWaves - 1) / kQWaves;
  const int blocks = (int)(blocks64 < kCosineBlocks ? (blocks64 > 0 ? blocks64 : 1) : kCosineBlocks);
  if (dtype == FB_BF16)
    hipLaunchKernelGGL(cosine_kernel<true>, dim3(blocks), dim3(kQThreads), 0, st,
                       static_cast<const char*>(a), static_cast<const char*>(b), rows, cols,
                       lda * elem, ldb * elem, partial);
  else
    hipLaunchKernelGGL(cosine_kernel<false>, dim3(blocks), dim3(kQThreads), 0, st,
                       static_cast<const char*>(a), static_cast<const char*>(b), rows, cols,
                       lda * elem, ldb * elem, partial);
  hipLaunchKernelGGL(mean_kernel, dim3(1), dim3(kQThreads), 0, st, partial, (int64_t)blocks * kQWaves,
                     rows, out);
  return hipGetLastError() == hipSuccess ? FB_OK : FB_EDEVICE;
}

// Rank loads of a replicated placement: slot value v = e + E * j is replica j of expert e, which
// carries floor(n_e / c_e) tokens plus one if j < n_e mod c_e (c_e = replicas of e).  One workgroup
// checks the placement rules (values in range, every expert present, the ordinals of every expert
// exactly 0 .. c_e - 1, no rank with two replicas of one expert, counts >= 0) and sums the shares per
// rank in LDS; a violated rule makes *max_mean = -1.  R * S <= FB_MAX_SLOTS_TOTAL and E <= R * S.
namespace {
__global__ __launch_bounds__(kQThreads) void slot_fold_kernel(
    const int32_t* __restrict__ counts, int32_t E, const int32_t* __restrict__ slots, int32_t R,
    int32_t S, int32_t* __restrict__ rank_loads, double* __restrict__ max_mean) {
  __shared__ int32_t reps[FB_MAX_SLOTS_TOTAL];   // replicas per expert
  __shared__ int32_t base[FB_MAX_SLOTS_TOTAL];   // exclusive prefix sum of reps
  __shared__ int32_t seen[FB_MAX_SLOTS_TOTAL];   // one flag per (expert, ordinal), at base[e] + j
  __shared__ int32_t sexp[FB_MAX_SLOTS_TOTAL];   // expert of every slot, -1 if empty or invalid
  __shared__ int32_t rl[FB_MAX_RANKS];
  __shared__ int32_t part[kQThreads];
  __shared__ int32_t s_bad;
  __shared__ long long s_mx[kQWaves], s_sum[kQWaves];
  const int tid = threadIdx.x;
  const int RS = R * S;
  if (tid == 0) s_bad = 0;
  for (int e = tid; e < E; e += kQThreads) reps[e] = 0;
  for (int c = tid; c < RS; c += kQThreads) seen[c] = 0;
  for (int r = tid; r < R; r += kQThreads) rl[r] = 0;
  __syncthreads();
  for (int c = tid; c < RS; c += kQThreads) {
    const int v = slots[c];
    int e = -1;
    if (v != -1) {
      if (v < 0 || v / E >= R) {
        s_bad = 1;
      } else {
        e = v % E;
        atomicAdd(&reps[e], 1);
      }
    }
    sexp[c] = e;
  }
  __syncthreads();
  // exclusive prefix sum of reps: each thread sums a contiguous chunk, thread 0 scans the chunks
  const int chunk = (E + kQThreads - 1) / kQThreads;
  const int e0 = tid * chunk, e1 = e0 + chunk < E ? e0 + chunk : E;
  int acc = 0;
  for (int e = e0; e < e1; ++e) acc += reps[e];
  part[tid] = acc;
  __syncthreads();
  if (tid == 0) {
    int run = 0;
    for (int t = 0; t < kQThreads; ++t) {
      const int x = part[t];
      part[t] = run;
      run += x;
    }
  }
  __syncthreads();
  acc = part[tid];
  for (int e = e0; e < e1; ++e) {
    base[e] = acc;
    acc += reps[e];
    if (reps[e] == 0 || counts[e] < 0) s_bad = 1;
  }
  __syncthreads();
  for (int c = tid; c < RS; c += kQThreads) {
    const int e = sexp[c];
    if (e < 0) continue;
    const int j = slots[c] / E;
    // base[e] + j stays below base[e] + reps[e] <= RS only when j < reps[e]
    if (j >= reps[e] || atomicAdd(&seen[base[e] + j], 1) != 0) {
      s_bad = 1;
      continue;
    }
    // no other slot of the same rank holds this expert
    const int r0 = (c / S) * S;
    for (int c2 = r0; c2 < c; ++c2)
      if (sexp[c2] == e) s_bad = 1;
    const int n = counts[e], k = reps[e];
    atomicAdd(&rl[c / S], n / k + (j < n % k ? 1 : 0));
  }
  __syncthreads();
  long long mx = 0, sum = 0;
  for (int r = tid; r < R; r += kQThreads) {
    const int v = rl[r];
    rank_loads[r] = v;
    mx = v > mx ? v : mx;
    sum += v;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const long long om = __shfl_xor(mx, off), os = __shfl_xor(sum, off);
    mx = om > mx ? om : mx;
    sum += os;
  }
  if ((tid & 63) == 0) { s_mx[tid >> 6] = mx; s_sum[tid >> 6] = sum; }
  __syncthreads();
  if (tid == 0) {
    for (int w = 1; w < kQWaves; ++w) { mx = s_mx[w] > mx ? s_mx[w] : mx; sum += s_sum[w]; }
    *max_mean = s_bad ? -1.0 : (sum == 0 ? 1.0 : (double)mx * (double)R / (double)sum);
  }
}
}  // namespace

int launch_fold(const int32_t* counts, int32_t E, const int32_t* e2r, int32_t R, int32_t* rank_loads,
                double* max_mean, void* stream) {
  (void)hipGetLastError();
  hipLaunchKernelGGL(fold_kernel, dim3(1), dim3(kQThreads), 0, static_cast<hipStream_t>(stream), counts,
                     E, e2r, R, rank_loads, max_mean);
  return hipGetLastError() == hipSuccess ? FB_OK : FB_EDEVICE;
}

int launch_slot_fold(const int32_t* counts, int32_t E, const int32_t* slots, int32_t R, int32_t S,
                     int32_t* rank_loads, double* max_mean, void* stream) {
  (void)hipGetLastError();
  hipLaunchKernelGGL(slot_fold_kernel, dim3(1), dim3(kQThreads), 0, static_cast<hipStream_t>(stream),
                     counts, E, slots, R, S, rank_loads, max_mean);
  return hipGetLastError() == hipSuccess ? FB_OK : FB_EDEVICE;
}

}  // namespace fb
