// Pooled-score top-k block mask for gfx950: a content-dependent producer of the block mask
// (Sec. II-B: dynamic sparse attention predicts block relevance from pooled Q/K features).
//
//   pool_kernel         block means of Q and K: each thread folds 8 channels of one block over
//                       its tokens in ascending order (IEEE float32, one rounding per addition,
//                       16-byte loads), then one correctly rounded division by the token count,
//                       and each block's maximum |mean| (as float bits: non-negative floats order
//                       like their bit patterns);
//   head_max_kernel     the per-head maximum over the block maxima (one workgroup per head and
//                       tensor; a global atomic max per block instead serialised 2,841 updates on
//                       each of 80 addresses and cost a quarter of the producer's time);
//   quant_kernel        int8 codes rint(mean * fl32(127 / max)), clamped to [-127, 127];
//   score_select_kernel one workgroup per ROWS query blocks of a head: exact int32 scores
//                       s_ij = sum_c qcode_i[c] kcode_j[c] (v_dot4_i32_i8) for every KV block j
//                       into LDS, then one wavefront per row, holding the row in registers,
//                       finds the k-th largest score by bisection over the integer range, keeps every larger score, the first
//                       equal scores in ascending j up to k, and the diagonal if asked, and
//                       writes the mask row.
// Every step is exact or a single float32 rounding in a fixed order, so the mask is the same bit
// for bit as a plain implementation of the same definition.

#pragma clang fp contract(off)

#include "common.h"
#include "producer_launch.h"
#include "wavealign.h"

namespace {

constexpr int kPoolThreads = 128;  // (256 took 4% longer: fewer, larger workgroups per CU)
constexpr int kRows = 4;          // query blocks per score_select workgroup
constexpr int kSelThreads = 256;  // 4 wavefronts, one row each

// amax[which][bh] = max over the head's blocks of bmax[which][bh][j]; one workgroup per (which, bh)
__global__ __launch_bounds__(256) void head_max_kernel(WaProducerLaunch a) {
  __shared__ uint32_t part[4];
  const int64_t wh = blockIdx.x;  // which * bh + bh
  const uint32_t* b = a.bmax + wh * a.mb;
  uint32_t mx = 0u;
  for (int j = threadIdx.x; j < a.mb; j += 256) mx = b[j] > mx ? b[j] : mx;
  for (int o = 32; o > 0; o >>= 1) {
    const uint32_t u = __shfl_xor(mx, o);
    mx = u > mx ? u : mx;
  }
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = mx;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t m = part[0];
    for (int w = 1; w < 4; ++w) m = part[w] > m ? part[w] : m;
    a.amax[wh] = m;
  }
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// grid.x covers bh * mb * (D / 8) threads; grid.y = 0 for Q, 1 for K. The D / 8 threads of one
// block are consecutive lanes of one wavefront.
template <int D>
__global__ __launch_bounds__(kPoolThreads) void pool_kernel(WaProducerLaunch a) {
  constexpr int G = D / 8;  // 8-channel groups per block
  const int which = blockIdx.y;
  const uint16_t* x = (const uint16_t*)(which ? a.k : a.q);
  const int64_t gid = (int64_t)blockIdx.x * kPoolThreads + threadIdx.x;
  const int64_t total = (int64_t)a.bh * a.mb * G;
  const bool active = gid < total;
  const int g = (int)(gid % G);
  const int64_t bj = gid / G;  // bh * mb + j
  uint32_t mx = 0u;
  if (active) {
    const int j = (int)(bj % a.mb);
    const int64_t bh = bj / a.mb;
    const int t0 = j * a.block;
    const int cnt = min(a.block, a.seq_len - t0);
    const uint16_t* p = x + ((int64_t)bh * a.seq_len + t0) * D + 8 * g;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    int t = 0;
    for (; t + 8 <= cnt; t += 8) {
      uint4 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = *(const uint4*)(p + (int64_t)(t + u) * D);
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        acc[0] += bf16_lo(v[u].x);
        acc[1] += bf16_hi(v[u].x);
        acc[2] += bf16_lo(v[u].y);
        acc[3] += bf16_hi(v[u].y);
        acc[4] += bf16_lo(v[u].z);
        acc[5] += bf16_hi(v[u].z);
        acc[6] += bf16_lo(v[u].w);
        acc[7] += bf16_hi(v[u].w);
      }
    }
    for (; t < cnt; ++t) {
      const uint4 v = *(const uint4*)(p + (int64_t)t * D);
      acc[0] += bf16_lo(v.x);
      acc[1] += bf16_hi(v.x);
      acc[2] += bf16_lo(v.y);
      acc[3] += bf16_hi(v.y);
      acc[4] += bf16_lo(v.z);
      acc[5] += bf16_hi(v.z);
      acc[6] += bf16_lo(v.w);
      acc[7] += bf16_hi(v.w);
    }
    const float c = (float)cnt;
    float* out = a.means + ((int64_t)which * a.bh * a.mb + bj) * D + 8 * g;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float m = acc[e] / c;
      out[e] = m;
      const uint32_t b = __float_as_uint(fabsf(m));
      mx = b > mx ? b : mx;
    }
  }
  // maximum over the G lanes of this block (every lane takes part)
#pragma unroll
  for (int o = G / 2; o > 0; o >>= 1) {
    const uint32_t u = __shfl_xor(mx, o);
    mx = u > mx ? u : mx;
  }
  if (active && g == 0) a.bmax[(int64_t)which * a.bh * a.mb + bj] = mx;
}

// codes[which][bh][mb][D] = rint(mean * fl32(127 / max)) clamped, 0 when max = 0
template <int D>
__global__ __launch_bounds__(256) void quant_kernel(WaProducerLaunch a) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t per = (int64_t)a.bh * a.mb * D;
  if (i >= 2 * per) return;
  const int64_t which = i / per;
  const int64_t bh = (i % per) / ((int64_t)a.mb * D);
  const float mx = __uint_as_float(a.amax[which * a.bh + bh]);
  int8_t code = 0;
  if (mx > 0.f) {
    const float inv = 127.0f / mx;
    float r = __builtin_rintf(a.means[i] * inv);
    r = fminf(fmaxf(r, -127.f), 127.f);
    code = (int8_t)(int)r;
  }
  a.codes[i] = code;
}

// One workgroup: query blocks [r0, r0 + kRows) of head bh.
template <int D>
__global__ __launch_bounds__(kSelThreads) void score_select_kernel(WaProducerLaunch a) {
  constexpr int W4 = D / 4;  // 32-bit words of one code row
  constexpr int JT = WA_MAX_BLOCKS / 64;  // scores of one row per lane
  extern __shared__ __attribute__((aligned(16))) int32_t sc[];  // [kRows][mb] scores
  __shared__ int32_t qs[kRows][W4];
  const int tiles = (a.mb + kRows - 1) / kRows;
  const int64_t bh = blockIdx.x / tiles;
  const int r0 = (int)(blockIdx.x % tiles) * kRows;
  const int nr = min(kRows, a.mb - r0);
  const int tid = threadIdx.x;
  const int mb = a.mb;
  const int32_t* qc = (const int32_t*)(a.codes + ((int64_t)bh * mb) * D);
  const int32_t* kc = (const int32_t*)(a.codes + ((int64_t)a.bh * mb + (int64_t)bh * mb) * D);
  for (int e = tid; e < kRows * W4; e += kSelThreads) {
    const int r = e / W4, w = e % W4;
    qs[r][w] = r < nr ? qc[(int64_t)(r0 + r) * W4 + w] : 0;
  }
  __syncthreads();
  // scores: one KV block per thread and pass
  for (int j = tid; j < mb; j += kSelThreads) {
    int32_t s[kRows];
#pragma unroll
    for (int r = 0; r < kRows; ++r) s[r] = 0;
    const int4* kr = (const int4*)(kc + (int64_t)j * W4);
#pragma unroll
    for (int w4 = 0; w4 < W4 / 4; ++w4) {
      const int4 kv = kr[w4];
      const int kw[4] = {kv.x, kv.y, kv.z, kv.w};
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int r = 0; r < kRows; ++r) s[r] = __builtin_amdgcn_sdot4(qs[r][4 * w4 + u], kw[u], s[r], false);
    }
#pragma unroll
    for (int r = 0; r < kRows; ++r) sc[r * mb + j] = s[r];
  }
  __syncthreads();
  // selection: wavefront w handles row w, with the row's scores in registers (entry t of lane l is
  // block 64 t + l; entries past the row hold INT32_MIN and are never counted)
  const int lane = tid & 63, r = tid >> 6;
  if (r >= nr) return;
  const int keep = a.keep < mb ? a.keep : mb;
  const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
  const int32_t* row = sc + r * mb;
  const int i = r0 + r;
  int32_t val[JT];
#pragma unroll
  for (int t = 0; t < JT; ++t) {
    const int j = 64 * t + lane;
    val[t] = j < mb ? row[j] : INT32_MIN;
  }
  // k-th largest value v: the largest v with #{s >= v} >= keep
  int lo = INT32_MAX, hi = INT32_MIN;
#pragma unroll
  for (int t = 0; t < JT; ++t)
    if (64 * t + lane < mb) {
      lo = min(lo, val[t]);
      hi = max(hi, val[t]);
    }
  for (int o = 32; o > 0; o >>= 1) {
    lo = min(lo, __shfl_xor(lo, o));
    hi = max(hi, __shfl_xor(hi, o));
  }
  // invariant: #{s >= lo} >= keep (lo = the minimum counts every entry), #{s >= hi + 1} < keep
  while (keep > 0 && lo < hi) {
    const int mid = lo + (int)(((int64_t)hi - lo + 1) / 2);
    int c = 0;
#pragma unroll
    for (int t = 0; t < JT; ++t) c += val[t] >= mid;
    for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o);
    if (c >= keep) lo = mid; else hi = mid - 1;
  }
  const int v = lo;
  int greater = 0;
#pragma unroll
  for (int t = 0; t < JT; ++t) greater += val[t] > v;
  for (int o = 32; o > 0; o >>= 1) greater += __shfl_xor(greater, o);
  const int ties = keep - greater;  // equal scores to keep, in ascending j
  uint8_t* out = a.mask + ((int64_t)bh * mb + i) * mb;
  int seen = 0;
#pragma unroll
  for (int t = 0; t < JT; ++t) {
    const int j = 64 * t + lane;
    const bool in = j < mb;
    const bool eq = in && keep > 0 && val[t] == v;
    const uint64_t eqw = __ballot(eq);
    const int rank = seen + __popcll(eqw & below);
    const bool kept = keep > 0 && in && (val[t] > v || (eq && rank < ties));
    const bool diag = a.diagonal && j == i;
    if (in) out[j] = (kept || diag) ? 1 : 0;
    seen += __popcll(eqw);
  }
}

}  // namespace

size_t wa_producer_select_smem(int mb) { return (size_t)kRows * mb * sizeof(int32_t); }

hipError_t wa_launch_producer(const WaProducerLaunch& a, hipStream_t stream) {
  if (a.bh <= 0 || a.mb <= 0) return hipSuccess;
  hipError_t e = hipSuccess;
  const int64_t pool_threads = (int64_t)a.bh * a.mb * (a.head_dim / 8);
  const dim3 pgrid((unsigned)((pool_threads + kPoolThreads - 1) / kPoolThreads), 2);
  const int64_t qn = 2ll * a.bh * a.mb * a.head_dim;
  const dim3 qgrid((unsigned)((qn + 255) / 256));
  const dim3 sgrid((unsigned)(a.bh * ((a.mb + kRows - 1) / kRows)));
  const size_t smem = wa_producer_select_smem(a.mb);
  if (a.head_dim == 128) {
    hipLaunchKernelGGL(pool_kernel<128>, pgrid, dim3(kPoolThreads), 0, stream, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(head_max_kernel, dim3((unsigned)(2 * a.bh)), dim3(256), 0, stream, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(quant_kernel<128>, qgrid, dim3(256), 0, stream, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = hipFuncSetAttribute((const void*)score_select_kernel<128>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                 (int)smem)) != hipSuccess)
      return e;
    hipLaunchKernelGGL(score_select_kernel<128>, sgrid, dim3(kSelThreads), smem, stream, a);
  } else if (a.head_dim == 64) {
    hipLaunchKernelGGL(pool_kernel<64>, pgrid, dim3(kPoolThreads), 0, stream, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(head_max_kernel, dim3((unsigned)(2 * a.bh)), dim3(256), 0, stream, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(quant_kernel<64>, qgrid, dim3(256), 0, stream, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = hipFuncSetAttribute((const void*)score_select_kernel<64>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                 (int)smem)) != hipSuccess)
      return e;
    hipLaunchKernelGGL(score_select_kernel<64>, sgrid, dim3(kSelThreads), smem, stream, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
