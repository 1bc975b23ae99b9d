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
//   score_select_kernel one workgroup per 16 query blocks of a head: exact int32 scores
//                       s_ij = sum_c qcode_i[c] kcode_j[c] with int8 MFMAs
//                       (v_mfma_i32_16x16x64_i8: 16 KV blocks x the 16 query blocks per
//                       instruction), 256 KV blocks per pass through a small LDS tile, so
//                       that each K code row is read once per 16 query blocks; each of the 16
//                       wavefronts collects one row's scores in registers, finds the k-th
//                       largest exactly by a radix select over 8-bit digits of the score minus
//                       the row minimum (one 256-bin LDS histogram per wavefront and digit),
//                       keeps every larger score, the first equal scores in ascending j up to
//                       k, and the diagonal if asked, and writes the row.
// Every step is exact or a single float32 rounding in a fixed order, so the mask is the same bit
// for bit as a plain implementation of the same definition.

#pragma clang fp contract(off)

#include "common.h"
#include "producer_launch.h"
#include "wavealign.h"

namespace {

constexpr int kPoolThreads = 128;  // (256 took 4% longer: fewer, larger workgroups per CU)
constexpr int kSelThreads = 1024;  // 16 wavefronts: one 16-KV-block tile each, then one row each
constexpr int kChunk = 256;        // KV blocks scored per pass (16 wavefronts x 16)

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

// Query blocks per score_select workgroup: RG groups of 16 (the MFMA's 16 columns), two when the
// rows' scores (2 JT registers) leave room for four wavefronts per SIMD, else one.
template <int JT>
struct SelGeom {
  static constexpr int RG = JT <= 48 ? 2 : 1;
  static constexpr int ROWS = 16 * RG;
};

// One workgroup: query blocks [r0, r0 + ROWS) of head bh. JT (a multiple of kChunk / 64 with
// 64 JT >= mb) is the number of scores of one row each lane holds.
template <int D, int JT>
__global__ __launch_bounds__(kSelThreads) void score_select_kernel(WaProducerLaunch a) {
  typedef int v4i __attribute__((ext_vector_type(4)));
  constexpr int RG = SelGeom<JT>::RG;
  constexpr int ROWS = SelGeom<JT>::ROWS;
  constexpr int KS = D / 64;                      // 64-channel steps of one MFMA each
  constexpr int NCH = JT * 64 / kChunk;           // passes over the KV blocks
  constexpr int CU = kChunk / 64;                 // entries per lane and pass
  __shared__ int32_t sc[ROWS][kChunk + 1];        // one pass's scores (+1: fewer bank conflicts)
  __shared__ int32_t hist[kSelThreads / 64][256];  // one digit histogram per wavefront
  __shared__ uint64_t rbits[kSelThreads / 64][JT];  // one row's kept bits per wavefront
  const int tiles = (a.mb + ROWS - 1) / ROWS;
  const int64_t bh = blockIdx.x / tiles;
  const int r0 = (int)(blockIdx.x % tiles) * ROWS;
  const int nr = min(ROWS, a.mb - r0);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int mb = a.mb;
  const int8_t* qc = a.codes + (bh * mb) * D;
  const int8_t* kc = a.codes + ((int64_t)a.bh * mb + bh * mb) * D;
  const v4i zero = {0, 0, 0, 0};
  // MFMA operands: lane l holds bytes [16 (l / 16), +16) of each 64-channel step of one code row,
  // row l mod 16 (the same channel split for both operands, so each product pairs equal channels).
  // B of group g: the Q codes of query block r0 + 16 g + l mod 16 (zero past the head).
  v4i qb[RG][KS];
#pragma unroll
  for (int g = 0; g < RG; ++g) {
    const int qr = r0 + 16 * g + (lane & 15);
#pragma unroll
    for (int st = 0; st < KS; ++st)
      qb[g][st] = qr < mb ? *(const v4i*)(qc + (int64_t)qr * D + 64 * st + 16 * (lane >> 4)) : zero;
  }
  // A of pass c: the K codes of KV block c kChunk + 16 w + l mod 16 (zero past the head), loaded
  // one pass ahead
  auto load_k = [&](int c, v4i (&ka)[KS]) {
    const int kv = c * kChunk + 16 * w + (lane & 15);
#pragma unroll
    for (int st = 0; st < KS; ++st)
      ka[st] = kv < mb ? *(const v4i*)(kc + (int64_t)kv * D + 64 * st + 16 * (lane >> 4)) : zero;
  };
  // the rows' scores: entry t of lane l is KV block 64 t + l; entries past the row hold INT32_MIN
  // and never count. Wavefront w collects query blocks r0 + w + 16 g. (NCH passes cover the row
  // exactly: kChunk (NCH - 1) < mb <= kChunk NCH, so every entry is written by its pass.)
  int32_t val[RG][JT];
  v4i ka[KS];
  load_k(0, ka);
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    v4i acc[RG];
#pragma unroll
    for (int g = 0; g < RG; ++g) {
      acc[g] = zero;
#pragma unroll
      for (int st = 0; st < KS; ++st) acc[g] = __builtin_amdgcn_mfma_i32_16x16x64_i8(ka[st], qb[g][st], acc[g], 0, 0, 0);
    }
    if (c + 1 < NCH) load_k(c + 1, ka);
    // each 16 x 16 result: lane l holds KV rows 4 (l / 16) + e, query column l mod 16 of its group
#pragma unroll
    for (int g = 0; g < RG; ++g)
#pragma unroll
      for (int e = 0; e < 4; ++e) sc[16 * g + (lane & 15)][16 * w + 4 * (lane >> 4) + e] = acc[g][e];
    __syncthreads();
#pragma unroll
    for (int g = 0; g < RG; ++g)
#pragma unroll
      for (int u = 0; u < CU; ++u) {
        const int j = c * kChunk + 64 * u + lane;
        val[g][c * CU + u] = j < mb ? sc[w + 16 * g][64 * u + lane] : INT32_MIN;
      }
    __syncthreads();  // every row is collected before the next pass overwrites the tile
  }
  const int keep = a.keep < mb ? a.keep : mb;
  const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
  for (int g = 0; g < RG; ++g) {
    if (w + 16 * g >= nr) break;
    const int i = r0 + w + 16 * g;
    const int32_t (&v_)[JT] = val[g];
    // (a score is at most 128 x 127 x 127 in magnitude, so INT32_MIN marks exactly the missing entries)
    int lo = INT32_MAX, hi = INT32_MIN;
#pragma unroll
    for (int t = 0; t < JT; ++t) {
      lo = min(lo, v_[t] == INT32_MIN ? INT32_MAX : v_[t]);
      hi = max(hi, v_[t]);
    }
    for (int o = 32; o > 0; o >>= 1) {
      lo = min(lo, __shfl_xor(lo, o));
      hi = max(hi, __shfl_xor(hi, o));
    }
    lo = __builtin_amdgcn_readfirstlane(lo);
    hi = __builtin_amdgcn_readfirstlane(hi);
    // The keep-th largest score, digit by digit of u = s - lo (0 <= u <= hi - lo < 2^23): at each
    // level the wavefront counts its candidates (entries whose higher digits equal the prefix found
    // so far) in 256 bins of the next 8 bits, and the bin holding the kept-th largest candidate fixes
    // those bits. Three levels resolve any row.
    // thr: the keep-th largest score; ties: how many scores equal to thr are kept (the first ones in
    // ascending j); neq: how many scores equal thr
    int thr = lo, ties = keep, neq = mb;  // all scores equal when lo == hi
    if (keep > 0 && lo < hi) {
      int32_t* h = hist[w];
      int nbits = 32 - __builtin_clz((uint32_t)(hi - lo));
      uint32_t prefix = 0u;
      int rem = keep;  // rank of the sought value among the candidates, from the top
      while (nbits > 0) {
        const int sh = nbits > 8 ? nbits - 8 : 0;
#pragma unroll
        for (int b = 0; b < 4; ++b) h[4 * lane + b] = 0;
        // (the wavefront's LDS operations complete in issue order; these fences keep that order)
        asm volatile("" ::: "memory");
#pragma unroll
        for (int t = 0; t < JT; ++t) {
          // below the prefix u wraps past 2^nbits; a missing entry (INT32_MIN) lands near 2^31
          const uint32_t u = (uint32_t)v_[t] - (uint32_t)lo - prefix;
          if ((u >> nbits) == 0u) atomicAdd(&h[u >> sh], 1);
        }
        asm volatile("" ::: "memory");
        int c[4];
#pragma unroll
        for (int b = 0; b < 4; ++b) c[b] = h[4 * lane + b];
        asm volatile("" ::: "memory");
        // candidates in the bins above this lane's four: suffix sum over the lanes
        const int tot = c[0] + c[1] + c[2] + c[3];
        int acc = tot;  // inclusive suffix sum: this lane and the lanes above it
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const int x = __shfl_down(acc, o);
          if (lane + o < 64) acc += x;
        }
        const int above = acc - tot;
        // bin 4 lane + b holds the rem-th largest candidate when above(b) < rem <= above(b) + c[b]
        int hit = -1, hit_above = 0, hit_cnt = 0;
        int ab = above;
#pragma unroll
        for (int b = 3; b >= 0; --b) {
          if (hit < 0 && ab < rem && rem <= ab + c[b]) {
            hit = 4 * lane + b;
            hit_above = ab;
            hit_cnt = c[b];
          }
          ab += c[b];
        }
        const uint64_t who = __ballot(hit >= 0);
        const int src = (int)__builtin_ctzll(who);
        const int bin = __builtin_amdgcn_readlane(hit, src);
        rem -= __builtin_amdgcn_readlane(hit_above, src);
        neq = __builtin_amdgcn_readlane(hit_cnt, src);  // at the last level (1-wide bins): the scores == thr
        prefix += (uint32_t)bin << sh;
        nbits = sh;
      }
      thr = lo + (int)prefix;
      ties = rem;  // the larger scores are keep - rem
    }
    // the row as bits, 64 blocks per word: word t = ballot of blocks 64 t .. 64 t + 63, kept by lane t
    uint64_t myword = 0ull;
    if (keep == 0 || ties == neq) {
      // every score >= thr is kept (a missing entry, INT32_MIN, is below any score)
#pragma unroll
      for (int t = 0; t < JT; ++t) {  // (words past the row come out 0)
        const uint64_t m = __ballot(keep > 0 && v_[t] >= thr);
        if (lane == t) myword = m;
      }
    } else {
      // only the first `ties` scores equal to thr, in ascending j
      int seen = 0;
#pragma unroll
      for (int t = 0; t < JT; ++t) {
        const uint64_t eqw = __ballot(v_[t] == thr);  // (past the row: INT32_MIN, never equal)
        const int rank = seen + __popcll(eqw & below);
        const uint64_t m = __ballot(v_[t] > thr || (v_[t] == thr && rank < ties));
        if (lane == t) myword = m;
        seen += __popcll(eqw);
      }
    }
    if (a.diagonal && lane == (i >> 6)) myword |= 1ull << (i & 63);
    const int nwords = (mb + 63) >> 6;
    uint64_t* rw = rbits[w];
    if (lane < nwords) rw[lane] = myword;
    asm volatile("" ::: "memory");  // (LDS operations of a wavefront complete in issue order)
    // Write the row's mb bytes: 16-byte stores of the 16-byte aligned chunks that lie inside the row,
    // single bytes at its two ends (the neighbouring rows' bytes belong to other wavefronts).
    uint8_t* out = a.mask + ((int64_t)bh * mb + i) * mb;
    const int off0 = (int)((uintptr_t)out & 15);
    uint8_t* g0 = out - off0;
    const int span = off0 + mb;
    for (int c = lane; 16 * c < span; c += 64) {
      const int b0 = 16 * c;
      if (b0 >= off0 && b0 + 16 <= span) {
        const int p0 = b0 - off0;  // row position of the chunk's first byte
        const int sh = p0 & 63;
        uint64_t x = rw[p0 >> 6] >> sh;
        if (sh > 48) x |= rw[(p0 >> 6) + 1] << (64 - sh);
        const uint32_t bits = (uint32_t)x;
        // 4 bits -> 4 bytes of 0 / 1: b * (1 + 2^7 + 2^14 + 2^21) puts bit e at bit 8 e (no carries)
        uint4 v;
        v.x = ((bits & 0xFu) * 0x204081u) & 0x01010101u;
        v.y = (((bits >> 4) & 0xFu) * 0x204081u) & 0x01010101u;
        v.z = (((bits >> 8) & 0xFu) * 0x204081u) & 0x01010101u;
        v.w = (((bits >> 12) & 0xFu) * 0x204081u) & 0x01010101u;
        *(uint4*)(g0 + b0) = v;
      } else {
        const int x0 = b0 > off0 ? b0 : off0;
        const int x1 = b0 + 16 < span ? b0 + 16 : span;
        for (int x = x0; x < x1; ++x) {
          const int pos = x - off0;
          g0[x] = (uint8_t)((rw[pos >> 6] >> (pos & 63)) & 1ull);
        }
      }
    }
    asm volatile("" ::: "memory");  // the next row's words are written after these reads
  }
}

template <int D, int JT>
hipError_t launch_select_t(const WaProducerLaunch& a, hipStream_t stream) {
  const dim3 grid((unsigned)(a.bh * ((a.mb + SelGeom<JT>::ROWS - 1) / SelGeom<JT>::ROWS)));
  hipLaunchKernelGGL((score_select_kernel<D, JT>), grid, dim3(kSelThreads), 0, stream, a);
  return hipGetLastError();
}

template <int D>
hipError_t launch_select(const WaProducerLaunch& a, hipStream_t stream) {
  const int jt = (a.mb + kChunk - 1) / kChunk * (kChunk / 64);  // scores per lane, whole passes
  if (jt <= 16) return launch_select_t<D, 16>(a, stream);
  if (jt <= 32) return launch_select_t<D, 32>(a, stream);
  if (jt <= 48) return launch_select_t<D, 48>(a, stream);
  return launch_select_t<D, WA_MAX_BLOCKS / 64>(a, stream);
}

template <int D>
hipError_t launch_all(const WaProducerLaunch& a, hipStream_t stream) {
  const int64_t pool_threads = (int64_t)a.bh * a.mb * (D / 8);
  const dim3 pgrid((unsigned)((pool_threads + kPoolThreads - 1) / kPoolThreads), 2);
  const int64_t qn = 2ll * a.bh * a.mb * D;
  const dim3 qgrid((unsigned)((qn + 255) / 256));
  hipError_t e;
  hipLaunchKernelGGL(pool_kernel<D>, pgrid, dim3(kPoolThreads), 0, stream, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(head_max_kernel, dim3((unsigned)(2 * a.bh)), dim3(256), 0, stream, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(quant_kernel<D>, qgrid, dim3(256), 0, stream, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return launch_select<D>(a, stream);
}

}  // namespace

hipError_t wa_launch_producer(const WaProducerLaunch& a, hipStream_t stream) {
  if (a.bh <= 0 || a.mb <= 0) return hipSuccess;
  if (a.mb > WA_MAX_BLOCKS) return hipErrorInvalidValue;
  if (a.head_dim == 128) return launch_all<128>(a, stream);
  if (a.head_dim == 64) return launch_all<64>(a, stream);
  return hipErrorInvalidValue;
}
