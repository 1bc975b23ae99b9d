// Pooled-score top-k block mask for gfx950: a content-dependent producer of the block mask
// (Sec. II-B: dynamic sparse attention predicts block relevance from pooled Q/K features).
//
// Three roles in one persistent kernel (one workgroup of 16 wavefronts per compute unit, taking
// items from one queue):
//   pooling     block means of Q and K: each thread folds 8 channels of one block over its
//               tokens in ascending order (IEEE float32, one rounding per addition, 16-byte
//               loads), then one correctly rounded division by the token count, and each
//               block's maximum |mean| (as float bits: non-negative floats order like their bit
//               patterns); an item is 64 blocks;
//   codes       per head and tensor, by the workgroup that pooled its last blocks: the head's
//               maximum over its block maxima, then int8 codes rint(mean * fl32(127 / max)),
//               clamped to [-127, 127];
//   selection   an item is 32 query blocks of a head (16 for rows of more than 3,072 blocks):
//               exact int32 scores s_ij = sum_c qcode_i[c] kcode_j[c] with int8 MFMAs
//               (v_mfma_i32_16x16x64_i8: 16 KV blocks x 16 query blocks per instruction),
//               256 KV blocks per pass through a small LDS tile, so that each K code row is
//               read once per 16 query blocks; each wavefront collects one row's scores in
//               registers, finds the k-th largest exactly by a radix select over 10-bit digits
//               of the score minus a floor under it (one 1,024-bin LDS histogram per wavefront and
//               digit), keeps every larger score, the first equal scores in ascending j up to
//               k, and the diagonal if asked, and writes the row.
// The heads are taken in groups of about 12,000 query blocks; step k of the queue holds the
// pooling of group k and the selection of group k - 2, interleaved, so that the memory-bound
// pooling of one group overlaps the compute-bound selection of another. A selection item waits
// for the codes of its head, whose pooling was queued two steps earlier. One launch replaces
// the earlier one launch per step, each of which ended with a partly idle chip.
// Every step is exact or a single float32 rounding in a fixed order, so the mask is the same bit
// for bit as a plain implementation of the same definition.

#pragma clang fp contract(off)

#include "common.h"
#include "producer_launch.h"
#include "wavealign.h"

namespace {

// Workgroup barrier that waits only for this wavefront's LDS operations (a full __syncthreads also
// waits for every global load in flight, which would drain the K-code load issued for the next
// pass); the compiler may not move memory accesses across it.
#define WA_LDS_BARRIER() asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory")

// Threads per workgroup, every role: 16 wavefronts, one workgroup per CU. 512 (two per CU, so that a
// pooling and a selection item can share one; 16-row selection items) took 1.64 ms per call
// against 1.52: the scoring passes then serve half as many rows each.
constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kWgPerCu = 1024 / kThreads;  // resident workgroups per compute unit (four wavefronts per SIMD)
constexpr int kChunk = 256;        // KV blocks scored per pass
constexpr int kKvTiles = kChunk / 16 / kWaves;  // 16-KV-block MFMA tiles per wavefront and pass
static_assert(kKvTiles >= 1 && kKvTiles * 16 * kWaves == kChunk, "a pass splits into whole tiles");
// Channels folded per pooling thread: 8 (one 16-byte load per token). 4 (8-byte loads, twice the
// threads) took 1.93 ms per call against 1.79, 16 (two loads per token) 2.67 (measured when the
// pipeline took one launch per step).
constexpr int kPoolCh = 8;
static_assert(kPoolCh == 8, "the pooling role stages its 8 means per lane as two float4");

// Stores that other workgroups of the same launch read (block means and maxima, head maxima,
// codes): device-scope atomic stores, which gfx950 writes through to the level every XCD sees, so
// that publishing them takes only a wait for their completion rather than a write-back of the
// whole L2 (the release fence on this multi-XCD chip).
template <typename T>
__device__ __forceinline__ void dev_store(T* p, T v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Lane moves through DPP (a few cycles, where a lane shuffle is an LDS round trip): lanes that the
// control leaves without a source, or that the row mask excludes, take `old`.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ int dpp32(int old, int v) {
  return __builtin_amdgcn_update_dpp(old, v, CTRL, ROW_MASK, 0xf, false);
}
// Minimum and maximum over the wavefront: xor 1 and 2 within quads, the half-row and row mirrors,
// then the broadcasts of lanes 15 and 31 into the rows above, which leave the result in lane 63.
__device__ __forceinline__ int wave_min(int v) {
  v = min(v, dpp32<0xB1, 0xf>(INT32_MAX, v));
  v = min(v, dpp32<0x4E, 0xf>(INT32_MAX, v));
  v = min(v, dpp32<0x141, 0xf>(INT32_MAX, v));
  v = min(v, dpp32<0x140, 0xf>(INT32_MAX, v));
  v = min(v, dpp32<0x142, 0xa>(INT32_MAX, v));
  v = min(v, dpp32<0x143, 0xc>(INT32_MAX, v));
  return __builtin_amdgcn_readlane(v, 63);
}
__device__ __forceinline__ int wave_max(int v) {
  v = max(v, dpp32<0xB1, 0xf>(INT32_MIN, v));
  v = max(v, dpp32<0x4E, 0xf>(INT32_MIN, v));
  v = max(v, dpp32<0x141, 0xf>(INT32_MIN, v));
  v = max(v, dpp32<0x140, 0xf>(INT32_MIN, v));
  v = max(v, dpp32<0x142, 0xa>(INT32_MIN, v));
  v = max(v, dpp32<0x143, 0xc>(INT32_MIN, v));
  return __builtin_amdgcn_readlane(v, 63);
}
// Inclusive prefix sum over the lanes: shifts by 1, 2, 4 and 8 within each row of 16, then the
// broadcasts of lane 15 into rows 1 and 3 and of lane 31 into rows 2 and 3.
__device__ __forceinline__ int lane_prefix_sum(int x) {
  x += dpp32<0x111, 0xf>(0, x);  // row_shr:1
  x += dpp32<0x112, 0xf>(0, x);  // row_shr:2
  x += dpp32<0x114, 0xf>(0, x);  // row_shr:4
  x += dpp32<0x118, 0xf>(0, x);  // row_shr:8
  x += dpp32<0x142, 0xa>(0, x);  // row_bcast:15
  x += dpp32<0x143, 0xc>(0, x);  // row_bcast:31
  return x;
}

// Pooling role of workgroup wg: threads wg * kThreads + tid cover Q, then K, of heads [h0, h0 + nh),
// D / kPoolCh consecutive threads (lanes of one wavefront) per block, each folding kPoolCh channels.
// stage: 2 KB of LDS private to the wavefront, through which its means are regrouped so that each
// store instruction writes 512 contiguous bytes (the stores go through to memory, so partly
// filled lines would be written more than once).
template <int D>
__device__ __forceinline__ void pool_role(const WaProducerLaunch& a, int h0, int nh, int64_t wg, int tid,
                                          float* stage) {
  constexpr int CH = kPoolCh;
  constexpr int G = D / CH;       // channel groups per block
  constexpr int U = 64 / CH;      // tokens per round of loads (128 bytes in flight per thread)
  typedef unsigned vec __attribute__((ext_vector_type(CH / 2)));
  const int64_t per = (int64_t)nh * a.mb * G;
  const int64_t gid = wg * kThreads + tid;
  const bool active = gid < 2 * per;
  const int which = gid < per ? 0 : 1;
  const uint16_t* x = (const uint16_t*)(which ? a.k : a.q);
  const int64_t rem = gid - which * per;
  const int g = (int)(rem % G);
  const int64_t bj = (int64_t)h0 * a.mb + rem / G;  // bh * mb + j
  uint32_t mx = 0u;
  if (active) {
    const int j = (int)(bj % a.mb);
    const int64_t bh = bj / a.mb;
    const int t0 = j * a.block;
    const int cnt = min(a.block, a.seq_len - t0);
    const uint16_t* p = x + ((int64_t)bh * a.seq_len + t0) * D + CH * g;
    float acc[CH];
#pragma unroll
    for (int e = 0; e < CH; ++e) acc[e] = 0.f;
    auto fold = [&](const vec& v) {
#pragma unroll
      for (int w = 0; w < CH / 2; ++w) {
        acc[2 * w] += bf16_lo(v[w]);
        acc[2 * w + 1] += bf16_hi(v[w]);
      }
    };
    int t = 0;
    for (; t + U <= cnt; t += U) {
      vec v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load((const vec*)(p + (int64_t)(t + u) * D));  // read once
#pragma unroll
      for (int u = 0; u < U; ++u) fold(v[u]);
    }
    for (; t < cnt; ++t) fold(*(const vec*)(p + (int64_t)t * D));
    const float c = (float)cnt;
#pragma unroll
    for (int e = 0; e < CH; ++e) {
      acc[e] = acc[e] / c;
      const uint32_t b = __float_as_uint(fabsf(acc[e]));
      mx = b > mx ? b : mx;
    }
    // lane l's channels are floats [8 l, 8 l + 8) of the wavefront's 512 (its 64 / G blocks in order)
    float4* st = (float4*)(stage + CH * (tid & 63));
    st[0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
    st[1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
  }
  asm volatile("" ::: "memory");  // (a wavefront's LDS operations complete in issue order)
  {
    // store k: floats [128 k + 2 l, +2) of the wavefront, block (128 k + 2 l) / D of its blocks
    const int lane = tid & 63;
    const int64_t lb0 = (wg * kThreads + (tid & ~63)) / G;  // the wavefront's first block
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int f = 128 * k + 2 * lane;
      const int64_t lb = lb0 + f / D;
      if (lb < 2ll * nh * a.mb) {
        const int wb = lb < (int64_t)nh * a.mb ? 0 : 1;
        const int64_t b_ = (int64_t)h0 * a.mb + lb - (int64_t)wb * nh * a.mb;
        const float2 v = *(const float2*)(stage + f);
        dev_store((uint64_t*)(a.means + ((int64_t)wb * a.bh * a.mb + b_) * D + f % D),
                  (uint64_t)__float_as_uint(v.x) | ((uint64_t)__float_as_uint(v.y) << 32));
      }
    }
  }
  // maximum over the G lanes of this block (every lane takes part; non-negative float bits compare
  // like integers): xor 1 and 2 within quads, the half-row mirror, and for 16 lanes the row mirror
  static_assert(G == 8 || G == 16, "a block's lanes are half a DPP row or a whole one");
  int m = (int)mx;
  m = max(m, dpp32<0xB1, 0xf>(0, m));
  m = max(m, dpp32<0x4E, 0xf>(0, m));
  m = max(m, dpp32<0x141, 0xf>(0, m));
  if (G == 16) m = max(m, dpp32<0x140, 0xf>(0, m));
  mx = (uint32_t)m;
  if (active && g == 0) dev_store(a.bmax + (int64_t)which * a.bh * a.mb + bj, mx);
}

// Codes role of one workgroup: head bh of Q (which = 0) or K (which = 1): the head's maximum block
// maximum, then codes rint(mean * fl32(127 / max)) clamped to [-127, 127], 0 when max = 0.
template <int D>
__device__ __forceinline__ void codes_role(const WaProducerLaunch& a, int which, int64_t bh, uint32_t* part,
                                           int tid) {
  const int64_t wh = which * (int64_t)a.bh + bh;
  const uint32_t* b = a.bmax + wh * a.mb;
  uint32_t mx = 0u;
  for (int j = tid; j < a.mb; j += kThreads) mx = b[j] > mx ? b[j] : mx;
  mx = (uint32_t)wave_max((int)mx);  // (non-negative float bits compare like integers)
  if ((tid & 63) == 0) part[tid >> 6] = mx;
  __syncthreads();
  uint32_t m = part[0];
  for (int w = 1; w < kThreads / 64; ++w) m = part[w] > m ? part[w] : m;
  if (tid == 0) dev_store(a.amax + wh, m);
  const float fmx = __uint_as_float(m);
  const float inv = fmx > 0.f ? 127.0f / fmx : 0.f;
  const float4* src = (const float4*)(a.means + wh * a.mb * D);
  uint32_t* dst = (uint32_t*)(a.codes + wh * a.mb * D);
  const int n4 = a.mb * D / 4;
  for (int e = tid; e < n4; e += kThreads) {
    const float4 v = src[e];
    uint32_t word = 0u;
    if (fmx > 0.f) {
      const float c[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float r = __builtin_rintf(c[q] * inv);
        r = fminf(fmaxf(r, -127.f), 127.f);
        word |= (uint32_t)(uint8_t)(int8_t)(int)r << (8 * q);
      }
    }
    dev_store(dst + e, word);
  }
}

// Bytes per Q code row in LDS: 128 + 16, so that the 16 rows one MFMA operand read takes lie in
// distinct banks.
constexpr int kQsStride = 144;

// Query blocks per selection item: RPW rows per wavefront (two when their scores, 2 JT registers,
// leave room for four wavefronts per SIMD, else one), in QG groups of the MFMA's 16 columns.
template <int JT>
struct SelGeom {
  static constexpr int RPW = JT <= 48 ? 2 : 1;
  static constexpr int ROWS = kWaves * RPW;
  static constexpr int QG = (ROWS + 15) / 16;
};

// Digits of the radix select: 10 bits (1,024 bins, 16 per lane), so that two levels resolve the
// score ranges of 16 to 19 bits seen in practice (8-bit digits took three passes over the row).
constexpr int kDigitBits = 10;
constexpr int kBins = 1 << kDigitBits;
constexpr int kBinsPerLane = kBins / 64;

// LDS of the kernel: the selection role's tiles; a pooling item stages its means in the score tile
// and the codes take their partial maxima from the histograms (items never overlap in a workgroup)
template <int JT>
struct SelLds {
  int32_t sc[2][16 * SelGeom<JT>::QG][kChunk + 1];  // scores of two passes in turn (+1: fewer bank conflicts)
  __attribute__((aligned(16))) int8_t qs[16 * SelGeom<JT>::QG][kQsStride];  // the rows' Q codes (d <= 128)
  __attribute__((aligned(16))) int32_t hist[kThreads / 64][kBins];  // one digit histogram per wavefront
  uint64_t rbits[kThreads / 64][JT];       // one row's kept bits per wavefront
};

static_assert(sizeof(SelLds<64>::sc) >= kThreads / 64 * 2048, "pooling stages 2 KB per wavefront in the score tile");

// Selection role of one workgroup: query blocks [r0, r0 + ROWS) of head bh. JT (a multiple of
// kChunk / 64 with 64 JT >= mb) is the number of scores of one row each lane holds.
template <int D, int JT>
__device__ __forceinline__ void select_role(const WaProducerLaunch& a, int64_t bh, int r0, SelLds<JT>& L, int tid) {
  typedef int v4i __attribute__((ext_vector_type(4)));
  constexpr int RPW = SelGeom<JT>::RPW;
  constexpr int ROWS = SelGeom<JT>::ROWS;
  constexpr int QG = SelGeom<JT>::QG;
  constexpr int KS = D / 64;                      // 64-channel steps of one MFMA each
  constexpr int NCH = JT * 64 / kChunk;           // passes over the KV blocks
  constexpr int CU = kChunk / 64;                 // entries per lane and pass
  const int nr = min(ROWS, a.mb - r0);
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int mb = a.mb;
  const int8_t* qc = a.codes + (bh * mb) * D;
  const int8_t* kc = a.codes + ((int64_t)a.bh * mb + bh * mb) * D;
  const v4i zero = {0, 0, 0, 0};
  // MFMA operands: lane l holds bytes [16 (l / 16), +16) of each 64-channel step of one code row,
  // row l mod 16 (the same channel split for both operands, so each product pairs equal channels).
  // B of group g: the Q codes of query block r0 + 16 g + l mod 16 (zero past the item or the
  // head), staged in LDS once and read there before each product (registers are the scarce
  // resource here).
  for (int e = tid; e < 16 * QG * (D / 16); e += kThreads) {
    const int row = e / (D / 16), col = e % (D / 16);
    const int qr = r0 + row;
    *(v4i*)&L.qs[row][16 * col] =
        row < ROWS && qr < mb ? *(const v4i*)(qc + (int64_t)qr * D + 16 * col) : zero;
  }
  // A of tile tt of pass c: the K codes of KV block c kChunk + 16 (kKvTiles w + tt) + l mod 16 (zero
  // past the head), loaded one pass ahead. Only the passes that reach past the head check (the
  // last one, and on short heads the ones after it).
  auto load_k = [&](int c, v4i (&ka)[kKvTiles][KS]) {
#pragma unroll
    for (int tt = 0; tt < kKvTiles; ++tt) {
      const int kv = c * kChunk + 16 * (kKvTiles * w + tt) + (lane & 15);
      const bool in = (c + 1) * kChunk <= mb || kv < mb;
#pragma unroll
      for (int st = 0; st < KS; ++st)
        ka[tt][st] = in ? *(const v4i*)(kc + (int64_t)kv * D + 64 * st + 16 * (lane >> 4)) : zero;
    }
  };
  // the rows' scores: entry t of lane l is KV block 64 t + l; entries past the row hold INT32_MIN
  // and never count. Wavefront w collects query blocks r0 + w + kWaves r. (mb <= kChunk NCH, so
  // every entry of the row is written by its pass.)
  int32_t val[RPW][JT];
  v4i ka[kKvTiles][KS];
  load_k(0, ka);
  WA_LDS_BARRIER();  // the Q codes are in LDS
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    v4i acc[kKvTiles][QG];
#pragma unroll
    for (int tt = 0; tt < kKvTiles; ++tt)
#pragma unroll
      for (int g = 0; g < QG; ++g) {
        acc[tt][g] = zero;
#pragma unroll
        for (int st = 0; st < KS; ++st) {
          const v4i qb = *(const v4i*)&L.qs[16 * g + (lane & 15)][64 * st + 16 * (lane >> 4)];
          acc[tt][g] = __builtin_amdgcn_mfma_i32_16x16x64_i8(ka[tt][st], qb, acc[tt][g], 0, 0, 0);
        }
      }
    if (c + 1 < NCH) load_k(c + 1, ka);
    // each 16 x 16 result: lane l holds KV rows 4 (l / 16) + e, query column l mod 16 of its group.
    // Passes alternate between two tiles: the barrier of pass c + 1 (every wavefront has collected
    // pass c) orders the reads of pass c before pass c + 2 overwrites that tile.
    int32_t (&sc)[16 * QG][kChunk + 1] = L.sc[c & 1];
#pragma unroll
    for (int tt = 0; tt < kKvTiles; ++tt)
#pragma unroll
      for (int g = 0; g < QG; ++g)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          sc[16 * g + (lane & 15)][16 * (kKvTiles * w + tt) + 4 * (lane >> 4) + e] = acc[tt][g][e];
    WA_LDS_BARRIER();
#pragma unroll
    for (int r = 0; r < RPW; ++r)
#pragma unroll
      for (int u = 0; u < CU; ++u) {
        const int j = c * kChunk + 64 * u + lane;
        const int x = sc[w + kWaves * r][64 * u + lane];  // (past the head: a product with zero codes)
        val[r][c * CU + u] = (c + 1) * kChunk <= mb || j < mb ? x : INT32_MIN;
      }
  }
  const int keep = a.keep < mb ? a.keep : mb;
  const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
  for (int r = 0; r < RPW; ++r) {
    if (w + kWaves * r >= nr) break;
    const int i = r0 + w + kWaves * r;
    const int32_t (&v_)[JT] = val[r];
    // (a score is at most 128 x 127 x 127 in magnitude, so INT32_MIN marks exactly the missing entries)
    int lo = INT32_MAX, hi = INT32_MIN;
#pragma unroll
    for (int t = 0; t < JT; ++t) {
      lo = min(lo, v_[t] == INT32_MIN ? INT32_MAX : v_[t]);
      hi = max(hi, v_[t]);
    }
    lo = wave_min(lo);
    hi = wave_max(hi);
    // A floor under the keep-th largest score: each lane splits its entries into three groups
    // (t mod 3) and takes the smallest of the three group maxima; the floor is the smallest of
    // those over the lanes whose groups all hold a score. Every such group has a score at or above
    // the floor, so when the groups number at least keep, so is the keep-th largest score; the
    // search below then counts only the scores at or above it (about a quarter of the row at 5%
    // density), and the histogram atomics stop piling up on the crowded middle bins.
    int base = lo;
    if (keep > 0 && keep <= 3 * 64 && lo < hi) {
      int g0 = INT32_MIN, g1 = INT32_MIN, g2 = INT32_MIN;
#pragma unroll
      for (int t = 0; t < JT; t += 3) {
        g0 = max(g0, v_[t]);
        if (t + 1 < JT) g1 = max(g1, v_[t + 1]);
        if (t + 2 < JT) g2 = max(g2, v_[t + 2]);
      }
      const bool full = g0 != INT32_MIN && g1 != INT32_MIN && g2 != INT32_MIN;
      const int n_full = __popcll(__ballot(full));
      const int f = wave_min(full ? min(g0, min(g1, g2)) : INT32_MAX);
      if (3 * n_full >= keep && f < hi) base = f;
    }
    // The keep-th largest score, digit by digit of u = s - base (0 <= u <= hi - base < 2^23): at
    // each level the wavefront counts its candidates (entries whose higher digits equal the prefix
    // found so far) in kBins bins of the next kDigitBits bits, and the bin holding the kept-th
    // largest candidate fixes those bits. Two levels resolve a range below 2^20, three any.
    // thr: the keep-th largest score; ties: how many scores equal to thr are kept (the first ones in
    // ascending j); neq: how many scores equal thr
    int thr = lo, ties = keep, neq = mb;  // all scores equal when lo == hi
    if (keep > 0 && lo < hi) {
      int32_t* h = L.hist[w];
      int nbits = 32 - __builtin_clz((uint32_t)(hi - base));
      uint32_t prefix = 0u;
      int rem = keep;  // rank of the sought value among the candidates, from the top
      while (nbits > 0) {
        const int sh = nbits > kDigitBits ? nbits - kDigitBits : 0;
        typedef int v4i_t __attribute__((ext_vector_type(4)));
        // lane l holds bins [kBinsPerLane (63 - l), +kBinsPerLane): the bins above a lane's are
        // those of the lanes below it, so a prefix sum over the lanes counts them
        v4i_t* h4 = (v4i_t*)(h + kBinsPerLane * (63 - lane));
#pragma unroll
        for (int q = 0; q < kBinsPerLane / 4; ++q) h4[q] = v4i_t{0, 0, 0, 0};
        // (the wavefront's LDS operations complete in issue order; these fences keep that order)
        asm volatile("" ::: "memory");
#pragma unroll
        for (int t = 0; t < JT; ++t) {
          // below the floor or the prefix u wraps past 2^nbits; a missing entry (INT32_MIN) lands
          // near 2^31
          const uint32_t u = (uint32_t)v_[t] - (uint32_t)base - prefix;
          if ((u >> nbits) == 0u) atomicAdd(&h[u >> sh], 1);
        }
        asm volatile("" ::: "memory");
        int c[kBinsPerLane];
#pragma unroll
        for (int q = 0; q < kBinsPerLane / 4; ++q) {
          const v4i_t x = h4[q];
          c[4 * q] = x[0];
          c[4 * q + 1] = x[1];
          c[4 * q + 2] = x[2];
          c[4 * q + 3] = x[3];
        }
        asm volatile("" ::: "memory");
        // candidates in the bins above this lane's: a prefix sum over the lanes
        int tot = 0;
#pragma unroll
        for (int b = 0; b < kBinsPerLane; ++b) tot += c[b];
        const int above = lane_prefix_sum(tot) - tot;
        // bin kBinsPerLane (63 - lane) + b holds the rem-th largest candidate when
        // above(b) < rem <= above(b) + c[b]
        int hit = -1, hit_above = 0, hit_cnt = 0;
        int ab = above;
#pragma unroll
        for (int b = kBinsPerLane - 1; b >= 0; --b) {
          if (hit < 0 && ab < rem && rem <= ab + c[b]) {
            hit = kBinsPerLane * (63 - lane) + b;
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
      thr = base + (int)prefix;
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
    uint64_t* rw = L.rbits[w];
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

// Queue words of one call (workspace, cleared by producer_init_kernel at the start of every call):
//   [0]                          the next item;
//   [1]                          set if a wait for codes ran out (see producer_kernel: it cannot;
//                                the call's status word reports it too);
//   [kQueueDone + x]             blocks of x = which * bh + head pooled so far (which: 0 Q, 1 K);
//   [kQueueDone + 2 bh + x]      nonzero once the codes of x are written.
constexpr int kQueueDone = 64;
// Sleeps of about 0.25 us between looks at a flag before a wait gives up (about one second).
constexpr uint32_t kWaitLimit = 1u << 22;

__global__ __launch_bounds__(256) void producer_init_kernel(uint32_t* queue, int64_t words, int32_t* status) {
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < words; e += (int64_t)gridDim.x * 256) queue[e] = 0u;
  if (status && blockIdx.x == 0 && threadIdx.x == 0) *status = 0;
}

// The call's work as one sequence of items, taken in order from the queue by resident
// workgroups. Step k (k = 0 .. ng + 1) holds the pooling items of head group k and the
// selection items of group k - 2, interleaved in proportion to their counts, so that the
// memory-bound pooling of one group overlaps the compute-bound selection of another.
struct ProducerPlan {
  int32_t per, ng, tiles;
  int64_t pool_full, pool_last;  // pooling items of a full group and of the last group
  int64_t total;                 // items of all steps
};

template <int D, int JT>
// (launch bounds: four wavefronts per SIMD, so 128 registers per lane and kWgPerCu workgroups per CU)
__global__ __launch_bounds__(kThreads, 4) void producer_kernel(WaProducerLaunch a, ProducerPlan pl) {
  constexpr int ROWS = SelGeom<JT>::ROWS;
  constexpr int G = D / kPoolCh;
  __shared__ SelLds<JT> lds;
  __shared__ int64_t s_item;
  __shared__ int32_t s_nrec, s_rec[kThreads / G];
  uint32_t* const ready = a.queue + kQueueDone + 2 * (int64_t)a.bh;
  for (;;) {
    // the thread index as a value the compiler cannot see through: what the roles derive from it
    // is recomputed per item instead of being hoisted out of this loop and held in registers
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    __syncthreads();  // the previous item is finished everywhere
    if (tid == 0) {
      s_item = (int64_t)atomicAdd(a.queue, 1u);
      s_nrec = 0;
    }
    __syncthreads();
    int64_t r = s_item;
    if (r >= pl.total) break;
    // step k of the item and its place r in that step
    int k = 0;
    int64_t P = 0, S = 0;
    for (; k < pl.ng + 2; ++k) {
      P = k < pl.ng ? (k == pl.ng - 1 ? pl.pool_last : pl.pool_full) : 0;
      S = k >= 2 ? (int64_t)min(pl.per, a.bh - (k - 2) * pl.per) * pl.tiles : 0;
      if (r < P + S) break;
      r -= P + S;
    }
    if (k == pl.ng + 2) break;  // (not reached: the steps hold exactly pl.total items)
    const int64_t s_before = r * S / (P + S), s_after = (r + 1) * S / (P + S);
    if (s_after > s_before) {
      // selection: wait until the codes of its head are written. The pooling of the head's group
      // came two steps earlier in the queue, so every item it needs was taken by a workgroup that
      // is running and never waits; the bound only turns an impossible hang into an error.
      const int head = (k - 2) * pl.per + (int)(s_before / pl.tiles);
      if (tid == 0) {
        uint32_t n = 0;
        while (!(__hip_atomic_load(ready + head, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) &&
                 __hip_atomic_load(ready + a.bh + head, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))) {
          __builtin_amdgcn_s_sleep(8);
          if (++n == kWaitLimit) {
            atomicOr(a.queue + 1, 1u);
            if (a.status) atomicOr(a.status, WA_PRODUCE_WAIT_EXPIRED);
            break;
          }
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");  // the codes another workgroup wrote
      }
      __syncthreads();
      select_role<D, JT>(a, head, (int)(s_before % pl.tiles) * ROWS, lds, tid);
      continue;
    }
    // pooling of items r - s_before of group k
    const int h0 = k * pl.per, nh = min(pl.per, a.bh - h0);
    const int64_t idx = r - s_before;
    pool_role<D>(a, h0, nh, idx, tid, (float*)&lds.sc[0][0][0] + 512 * (tid >> 6));
    // publish: every wavefront's means and maxima (device-scope stores) have completed, then count
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (tid == 0) {
      // the item's blocks, by (tensor, head): blocks [b0, b1) of the group's 2 nh mb, in runs of one head
      const int64_t b0 = idx * (kThreads / G);
      const int64_t b1 = min(b0 + kThreads / G, 2ll * nh * a.mb);
      for (int64_t b = b0; b < b1;) {
        const int64_t x = b / a.mb;  // which * nh + local head
        const int64_t e = min(b1, (x + 1) * a.mb);
        const uint32_t cnt = (uint32_t)(e - b);
        const int which = (int)(x / nh);
        const int64_t wh = (int64_t)which * a.bh + h0 + x % nh;
        if (atomicAdd(a.queue + kQueueDone + wh, cnt) + cnt == (uint32_t)a.mb) s_rec[s_nrec++] = (int32_t)wh;
        b = e;
      }
      if (s_nrec > 0) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");  // the other workgroups' means
    }
    __syncthreads();
    // the workgroup that pooled the last blocks of a head and tensor writes its codes
    const int nrec = s_nrec;
    for (int q = 0; q < nrec; ++q) {
      const int wh = s_rec[q];
      codes_role<D>(a, wh / a.bh, wh % a.bh, (uint32_t*)lds.hist, tid);
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the codes (device-scope stores) are complete
      __syncthreads();
      if (tid == 0) dev_store(ready + wh, 1u);
    }
  }
}

// Query blocks per head group: about 12,000 (four heads of 2,841 blocks). Two-head groups took
// 1.78 ms per call against 1.74 for four (measured before the stores were made device-scope),
// one-head groups 2.06 ms: selections then reach their head before its codes are written.
constexpr int kGroupBlocks = 12000;

int producer_resident_cus() {
  static int cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cached[dev] <= 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

template <int D, int JT>
hipError_t launch_all_t(const WaProducerLaunch& a, hipStream_t stream) {
  const int per_blocks = (kGroupBlocks + a.mb / 2) / a.mb;
  ProducerPlan pl{};
  pl.per = per_blocks < 1 ? 1 : (per_blocks > a.bh ? a.bh : per_blocks);
  pl.ng = (a.bh + pl.per - 1) / pl.per;
  pl.tiles = (a.mb + SelGeom<JT>::ROWS - 1) / SelGeom<JT>::ROWS;
  constexpr int G = D / kPoolCh;
  auto pool_items = [&](int nh) { return (2ll * nh * a.mb * G + kThreads - 1) / kThreads; };
  const int last = a.bh - (pl.ng - 1) * pl.per;
  pl.pool_full = pool_items(pl.per);
  pl.pool_last = pool_items(last);
  pl.total = (pl.ng - 1) * pl.pool_full + pl.pool_last + (int64_t)a.bh * pl.tiles;
  const int64_t words = wa_producer_queue_words(a.bh);
  const int64_t init_wgs = (words + 255) / 256 < 1024 ? (words + 255) / 256 : 1024;
  hipLaunchKernelGGL(producer_init_kernel, dim3((unsigned)init_wgs), dim3(256), 0, stream, a.queue, words,
                     a.status);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t slots = (int64_t)producer_resident_cus() * kWgPerCu;
  const int64_t grid = pl.total < slots ? pl.total : slots;
  hipLaunchKernelGGL((producer_kernel<D, JT>), dim3((unsigned)grid), dim3(kThreads), 0, stream, a, pl);
  return hipGetLastError();
}

template <int D>
hipError_t launch_all(const WaProducerLaunch& a, hipStream_t stream) {
  const int jt = (a.mb + kChunk - 1) / kChunk * (kChunk / 64);  // scores per lane, whole passes
  if (jt <= 16) return launch_all_t<D, 16>(a, stream);
  if (jt <= 32) return launch_all_t<D, 32>(a, stream);
  if (jt <= 48) return launch_all_t<D, 48>(a, stream);
  return launch_all_t<D, WA_MAX_BLOCKS / 64>(a, stream);
}

}  // namespace

hipError_t wa_launch_producer(const WaProducerLaunch& a, hipStream_t stream) {
  if (a.bh <= 0 || a.mb <= 0) return hipSuccess;
  if (a.mb > WA_MAX_BLOCKS) return hipErrorInvalidValue;
  if (a.head_dim == 128) return launch_all<128>(a, stream);
  if (a.head_dim == 64) return launch_all<64>(a, stream);
  return hipErrorInvalidValue;
}
