// Cache-aware query-row permutation for gfx950.
//
// Phases (Sec. IV-C..IV-E, Alg. 1, Alg. 2):
//   0  mask statistics from the bit-packed rows and columns (n_i, c_j, nnz,
//      distinct columns, adjacent-row overlap, sum c_j^2);
//   1  skip cases 1-3 (fits in cache, too little work, already local);
//   2  matrix-free centred subspace iteration in exact fixed point: the centred
//      products are exact integer products of the packed mask with X (or Ys)
//      plus the rank-one centring corrections scaled by m (Alg. 1); the
//      2-column QR is a Cholesky-QR of the exactly summed Gram matrix (one IEEE
//      fp64 rounding per operation, no contraction); then Rayleigh-Ritz with
//      one Jacobi rotation and a canonical column sign;
//   3  skip case 4 (the rank-2 embedding keeps too little of ||M~||_F^2);
//   4  Stage 1: sort of the rows by polar angle (Eq. 4) with an exact
//      integer comparator (half-plane class, then the sign of the cross product,
//      then the row index);
//   5  Stage 2: the order is cut into n_xcd contiguous segments of equal work
//      (w_i = n_i + 1, a prefix sum over the order decides each row's segment)
//      and each segment into buckets of W rows; one bitonic sort over
//      (bucket, -n_i, position) keys sorts every bucket by descending n_i,
//      stably. The segment table is an output: the attention kernel runs
//      segment x on XCD x.
// Two forms, both exact, so the same result bit for bit:
//   * heads of at most 1024 rows and columns: perm_mfma_kernel, one 1024-thread workgroup per head
//     and one launch for all heads; the centred products are int8 matrix-core products of the
//     mask bits with the base-256 digits of X and Ys (see the kernel);
//   * larger heads: phases 0-1 and the first QR in perm_init_kernel, each further QR in
//     orth_step_kernel and phases 3-5 in perm_finish_kernel (one 1024-thread workgroup per head
//     each); the centred products, with the same matrix-core products, in mfma_gather_kernel and
//     mfma_scatter_kernel, one workgroup per 128 lines of every head. Per-head state between the
//     kernels lives in the workspace.
// Every sum is an exact integer, so neither the order of parallel reductions nor the slicing nor the
// form matters. Supports m, n <= 4096.

#pragma clang fp contract(off)

#include "common.h"
#include "perm_launch.h"

namespace {

constexpr int NT = 1024;
constexpr int NWAVE = NT / 64;
constexpr int MAXB = 4096;

constexpr int FLAG_FITS_CACHE = 1, FLAG_LITTLE_WORK = 2, FLAG_LOCAL = 4, FLAG_UNSTRUCTURED = 8, FLAG_DEGENERATE = 16,
              FLAG_IDENTITY = 64;
constexpr int SKIP_AUTO = 0, SKIP_ALWAYS = 2;

constexpr int PER = MAXB / NT;  // rows or columns per thread

struct Shared {
  int32_t cc[MAXB];          // column counts; later the Stage-1 order
  int32_t xs[2 * MAXB];      // X (2^30 fixed point), later U
  int32_t ys[2 * MAXB];      // sort scratch (indices, then 64-bit keys)
  int64_t red[NWAVE * 4];
  int32_t part[NT];          // scan partials
  int32_t seg[65];           // XCD segment starts of the current order
  double dbl[8];
  int64_t i64[8];
  int32_t i32[8];
};

__device__ __forceinline__ uint64_t splitmix64(uint64_t x) {
  uint64_t z = x + 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__device__ __forceinline__ int bitlen_u64(uint64_t v) { return v ? 64 - __clzll((long long)v) : 0; }
__device__ __forceinline__ uint64_t uabs64(int64_t v) { return v < 0 ? (uint64_t)(-v) : (uint64_t)v; }

// Wavefront reductions with DPP lane moves (a few cycles each, where a lane shuffle goes through
// LDS): xor 1 and xor 2 within quads, then the half-row and row mirrors, then the row broadcasts of
// lane 15 and lane 31, which leave the total in lane 63; it is read back to every lane.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint64_t dpp64(uint64_t v) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)v, CTRL, ROW_MASK, 0xf, false);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(v >> 32), CTRL, ROW_MASK, 0xf, false);
  return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ uint64_t lane63(uint64_t v) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, 63);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), 63);
  return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ int64_t wave_sum(int64_t v) {
  uint64_t u = (uint64_t)v;  // two's complement: the sum modulo 2^64 is the exact sum
  u += dpp64<0xB1, 0xf>(u);   // quad_perm [1,0,3,2]
  u += dpp64<0x4E, 0xf>(u);   // quad_perm [2,3,0,1]
  u += dpp64<0x141, 0xf>(u);  // row_half_mirror
  u += dpp64<0x140, 0xf>(u);  // row_mirror
  u += dpp64<0x142, 0xa>(u);  // row_bcast15 into rows 1 and 3
  u += dpp64<0x143, 0xc>(u);  // row_bcast31 into rows 2 and 3
  return (int64_t)lane63(u);
}
__device__ __forceinline__ uint64_t max64(uint64_t a, uint64_t b) { return a > b ? a : b; }
__device__ __forceinline__ uint64_t wave_max(uint64_t v) {
  v = max64(v, dpp64<0xB1, 0xf>(v));
  v = max64(v, dpp64<0x4E, 0xf>(v));
  v = max64(v, dpp64<0x141, 0xf>(v));
  v = max64(v, dpp64<0x140, 0xf>(v));
  v = max64(v, dpp64<0x142, 0xa>(v));
  v = max64(v, dpp64<0x143, 0xc>(v));
  return lane63(v);
}

// Sum of up to 4 int64 values over the workgroup; the result is returned to every thread.
template <int K>
__device__ void block_sum(Shared& sh, int64_t (&v)[K]) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int k = 0; k < K; ++k) v[k] = wave_sum(v[k]);
  if (lane == 0)
#pragma unroll
    for (int k = 0; k < K; ++k) sh.red[w * 4 + k] = v[k];
  __syncthreads();
#pragma unroll
  for (int k = 0; k < K; ++k) {
    int64_t s = 0;
    for (int i = 0; i < NWAVE; ++i) s += sh.red[i * 4 + k];
    v[k] = s;
  }
  __syncthreads();
}

__device__ uint64_t block_max(Shared& sh, uint64_t v) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  v = wave_max(v);
  if (lane == 0) sh.red[w * 4] = (int64_t)v;
  __syncthreads();
  uint64_t r = 0;
  for (int i = 0; i < NWAVE; ++i) {
    uint64_t u = (uint64_t)sh.red[i * 4];
    r = u > r ? u : r;
  }
  __syncthreads();
  return r;
}

struct Head {
  const uint64_t* rowbits;  // [nw][m] word-major: word w of row i at w * m + i
  const uint64_t* colbits;  // [mw][n] word-major: word v of column j at v * n + j
  const int32_t* row_nnz;   // [m]
  int m, n, nw, mw;
};

// Cholesky factor of the 2 x 2 Gram matrix g of a block Z (exact sums of its entries shifted to 24
// bits): r11, r12, r22, and whether the second column keeps a direction of its own (its residual u
// above G22 2^-30). One IEEE fp64 rounding per operation, no contraction.
struct Chol {
  double r11, r12, r22;
  bool rank2;
};
__device__ __forceinline__ Chol chol2(const int64_t (&g)[3]) {
  const double G11 = (double)g[0], G12 = (double)g[1], G22 = (double)g[2];
  Chol c;
  c.r11 = __builtin_sqrt(G11);
  c.r12 = G12 / c.r11;
  const double u = G22 - c.r12 * c.r12;
  c.rank2 = u > G22 * 0x1p-30;
  c.r22 = c.rank2 ? __builtin_sqrt(u) : 0.0;
  return c;
}

// Row (x0, x1) of the orthonormal factor X = Z R^-1 in 2^30 fixed point, from the row of Z shifted
// right by the Gram shift (z0s, z1s); the second entry is 0 when Z has rank one.
__device__ __forceinline__ void orth_row(const Chol& c, int64_t z0s, int64_t z1s, int32_t& x0, int32_t& x1) {
  const double q0 = (double)z0s / c.r11;
  x0 = (int32_t)__builtin_rint(q0 * 1073741824.0);
  if (c.rank2) {
    const double q1 = ((double)z1s - c.r12 * q0) / c.r22;
    x1 = (int32_t)__builtin_rint(q1 * 1073741824.0);
  } else {
    x1 = 0;
  }
}

// Cholesky-QR of Z (thread-owned rows i = tid + k NT, zr[k]) into sh.xs; true if degenerate.
__device__ bool orth(Shared& sh, const Head& H, const int64_t (&zr)[PER][2]) {
  const int tid = threadIdx.x;
  uint64_t mx = 0;
#pragma unroll
  for (int k = 0; k < PER; ++k)
    if (tid + k * NT < H.m) {
      const uint64_t a = uabs64(zr[k][0]), b = uabs64(zr[k][1]);
      mx = a > mx ? a : mx;
      mx = b > mx ? b : mx;
    }
  mx = block_max(sh, mx);
  const int bl = bitlen_u64(mx);
  const int s = bl > 24 ? bl - 24 : 0;
  int64_t g[3] = {0, 0, 0};
#pragma unroll
  for (int k = 0; k < PER; ++k)
    if (tid + k * NT < H.m) {
      const int64_t z0 = zr[k][0] >> s, z1 = zr[k][1] >> s;
      g[0] += z0 * z0;
      g[1] += z0 * z1;
      g[2] += z1 * z1;
    }
  block_sum<3>(sh, g);
  if (g[0] == 0) return true;
  if (tid == 0) {
    const Chol c = chol2(g);
    sh.dbl[0] = c.r11;
    sh.dbl[1] = c.r12;
    sh.dbl[2] = c.r22;
    sh.i32[0] = c.rank2 ? 1 : 0;
  }
  __syncthreads();
  const Chol c = {sh.dbl[0], sh.dbl[1], sh.dbl[2], sh.i32[0] != 0};
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int i = tid + k * NT;
    if (i < H.m) orth_row(c, zr[k][0] >> s, zr[k][1] >> s, sh.xs[2 * i], sh.xs[2 * i + 1]);
  }
  __syncthreads();
  return false;
}

// Threads that share one column (or row) in the one-workgroup form: the largest power of two up to
// 16 with threads * lines <= NT. They are consecutive lanes of one wavefront, and each takes a
// contiguous chunk of the line's bit range (or of the compared elements).
__device__ __forceinline__ int lanes_per_line(int lines) {
  int t = 1;
  while (t < 16 && 2 * t * lines <= NT) t *= 2;
  return t;
}

// Sum of an int64 over groups of t consecutive lanes (t a power of two up to 64); every lane of a
// group receives its group's sum.
__device__ __forceinline__ int64_t group_sum(int64_t v, int t) {
  for (int o = 1; o < t; o <<= 1) {
    const int lo = __shfl_xor((int)(uint32_t)(uint64_t)v, o);
    const int hi = __shfl_xor((int)(uint32_t)((uint64_t)v >> 32), o);
    v += (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint64_t)(uint32_t)lo);
  }
  return v;
}

// Heads of at most this many rows are ordered by rank sorts (no barriers; four or more lanes per
// row), larger ones by bitonic sorts (at 394 rows the rank sort's m^2 / 2 compares per lane cost
// more than the bitonic stages).
constexpr int kRankSortMax = 256;

// Z of the thread's rows (rows i = tid + k NT) as the product kernels wrote it.
__device__ void load_z(const WaPermLaunch& a, int h, int64_t (&zr)[PER][2]) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int i = tid + k * NT;
    zr[k][0] = i < a.m ? a.z[((int64_t)h * a.m + i) * 2] : 0;
    zr[k][1] = i < a.m ? a.z[((int64_t)h * a.m + i) * 2 + 1] : 0;
  }
}

__device__ __forceinline__ Head head_of(const WaPermLaunch& a, int h) {
  Head H;
  H.m = a.m;
  H.n = a.n;
  H.nw = (a.n + 63) / 64;
  H.mw = (a.m + 63) / 64;
  H.rowbits = a.rowbits + (int64_t)h * a.m * H.nw;
  H.colbits = a.colbits + (int64_t)h * a.n * H.mw;
  H.row_nnz = a.row_nnz + (int64_t)h * a.m;
  return H;
}

__device__ void store_x(const WaPermLaunch& a, const Shared& sh, int h) {
  int2* xg = reinterpret_cast<int2*>(a.xg) + (int64_t)h * a.m;
  for (int i = threadIdx.x; i < a.m; i += NT) xg[i] = make_int2(sh.xs[2 * i], sh.xs[2 * i + 1]);
}

__device__ __forceinline__ int angle_class(int64_t x, int64_t y) {
  if (y < 0) return 0;
  if (y == 0) return x >= 0 ? 1 : 3;
  return 2;
}

// true if row a precedes row b in ascending polar angle (ties: smaller index); -1 is +infinity
__device__ __forceinline__ bool angle_less(const Shared& sh, int a, int b) {
  if (a < 0) return false;
  if (b < 0) return true;
  const int64_t xa = sh.xs[2 * a], ya = sh.xs[2 * a + 1];
  const int64_t xb = sh.xs[2 * b], yb = sh.xs[2 * b + 1];
  const int ca = angle_class(xa, ya), cb = angle_class(xb, yb);
  if (ca != cb) return ca < cb;
  if (ca == 0 || ca == 2) {
    const int64_t cross = xa * yb - ya * xb;
    if (cross != 0) return cross > 0;
  }
  return a < b;
}

// The same order on (x, y, row) entries; row -1 is +infinity.
__device__ __forceinline__ bool entry_less(const int4& a, const int4& b) {
  if (a.z < 0) return false;
  if (b.z < 0) return true;
  const int ca = angle_class(a.x, a.y), cb = angle_class(b.x, b.y);
  if (ca != cb) return ca < cb;
  if (ca == 0 || ca == 2) {
    const int64_t cross = (int64_t)a.x * b.y - (int64_t)a.y * b.x;
    if (cross != 0) return cross > 0;
  }
  return a.z < b.z;
}

// Work-balanced XCD segments of the order held in sh.cc[0..m): position p belongs to segment
// min(n_xcd - 1, n_xcd * W_p / W_m) with W_p the sum of (n_i + 1) over the first p positions.
// Fills sh.seg[0..n_xcd] (and seg_out, if given). Uses sh.xs as scratch.
__device__ void compute_segments(Shared& sh, const int32_t* row_nnz, int m, int n_xcd, int32_t* seg_out) {
  const int tid = threadIdx.x;
  const int per = (m + NT - 1) / NT;
  const int lo = min(tid * per, m), hi = min(lo + per, m);
  int32_t local = 0;
  for (int p = lo; p < hi; ++p) local += row_nnz[sh.cc[p]] + 1;
  // prefix sums of the thread totals: within the wavefront by lane shifts, then over the wavefront totals
  const int lane = tid & 63, w = tid >> 6;
  int32_t incl = local;
  for (int o = 1; o < 64; o <<= 1) {
    const int32_t y = __shfl_up(incl, o);
    if (lane >= o) incl += y;
  }
  if (lane == 63) sh.part[w] = incl;
  __syncthreads();
  int32_t before = 0, sum = 0;
  for (int i = 0; i < NWAVE; ++i) {
    const int32_t t = sh.part[i];
    before += i < w ? t : 0;
    sum += t;
  }
  const int64_t total = sum;
  int32_t run = before + incl - local;   // W_lo
  int32_t* segof = sh.xs;
  for (int p = lo; p < hi; ++p) {
    const int64_t x = ((int64_t)n_xcd * run) / total;
    segof[p] = (int32_t)(x < n_xcd - 1 ? x : n_xcd - 1);
    run += row_nnz[sh.cc[p]] + 1;
  }
  __syncthreads();
  for (int p = tid; p < m; p += NT) {
    const int prev = p > 0 ? segof[p - 1] : -1;
    for (int x = prev + 1; x <= segof[p]; ++x) sh.seg[x] = p;
  }
  if (tid == 0)
    for (int x = segof[m - 1] + 1; x <= n_xcd; ++x) sh.seg[x] = m;
  __syncthreads();
  if (seg_out)
    for (int x = tid; x <= n_xcd; x += NT) seg_out[x] = sh.seg[x];
}

// Writes the identity order for head h (and its segments and flags).
__device__ void write_identity(const WaPermLaunch& a, Shared& sh, int h, int flags, bool zero_embedding) {
  const int tid = threadIdx.x, m = a.m;
  int32_t* perm = a.perm + (int64_t)h * m;
  for (int i = tid; i < m; i += NT) {
    perm[i] = i;
    sh.cc[i] = i;
    if (a.stage1) a.stage1[(int64_t)h * m + i] = i;
    if (zero_embedding && a.embedding) {
      a.embedding[((int64_t)h * m + i) * 2] = 0;
      a.embedding[((int64_t)h * m + i) * 2 + 1] = 0;
    }
  }
  __syncthreads();
  compute_segments(sh, a.row_nnz + (int64_t)h * m, m, a.n_xcd,
                   a.seg_start ? a.seg_start + (int64_t)h * (a.n_xcd + 1) : nullptr);
  if (a.flags && tid == 0) a.flags[h] = (uint8_t)(flags | FLAG_IDENTITY);
}

// What the set-up of a head leaves for the subspace iteration (uniform over the workgroup).
struct HeadInit {
  int status;  // 0: iterate; 1: done (statistics only, or a skipped head with its identity order written);
               // 2: the start block is degenerate
  int flags;   // skip-rule flags of cases 1-3
  int64_t nnz, sum_c2;
  int64_t adj_and, adj_or;  // adjacent-row overlap of the natural order
};
constexpr int HEAD_ITERATE = 0, HEAD_DONE = 1, HEAD_DEGENERATE = 2;

// Statistics, skip cases 1-3, and the first QR of the seeded start block (into sh.xs and a.xg).
__device__ HeadInit init_head(const WaPermLaunch& a, Shared& sh, int h) {
  const int tid = threadIdx.x;
  const int m = a.m, n = a.n;
  const Head H = head_of(a, h);

  // ---- phase 0: statistics ----
  // The word loops load 8 words at a time, so that their latencies overlap.
  constexpr int WB = 8;
  int64_t st[4] = {0, 0, 0, 0};  // nnz, distinct, sum c^2, (unused)
  for (int j = tid; j < n; j += NT) {
    int c = 0;
    for (int v0 = 0; v0 < H.mw; v0 += WB) {
      uint64_t wd[WB];
#pragma unroll
      for (int u = 0; u < WB; ++u) wd[u] = v0 + u < H.mw ? H.colbits[(int64_t)(v0 + u) * n + j] : 0ull;
#pragma unroll
      for (int u = 0; u < WB; ++u) c += __popcll(wd[u]);
    }
    a.cc[(int64_t)h * n + j] = c;
    if (a.col_cnt) a.col_cnt[(int64_t)h * n + j] = c;
    st[1] += c > 0;
    st[2] += (int64_t)c * c;
  }
  for (int i = tid; i < m; i += NT) st[0] += H.row_nnz[i];
  int64_t adj[2] = {0, 0};  // rows i and i + 1, word by word
  for (int i = tid; i < m - 1; i += NT) {
    for (int w0 = 0; w0 < H.nw; w0 += WB) {
      uint64_t x[WB], y[WB];
#pragma unroll
      for (int u = 0; u < WB; ++u) {
        x[u] = w0 + u < H.nw ? H.rowbits[(int64_t)(w0 + u) * m + i] : 0ull;
        y[u] = w0 + u < H.nw ? H.rowbits[(int64_t)(w0 + u) * m + i + 1] : 0ull;
      }
#pragma unroll
      for (int u = 0; u < WB; ++u) {
        adj[0] += __popcll(x[u] & y[u]);
        adj[1] += __popcll(x[u] | y[u]);
      }
    }
  }
  block_sum<4>(sh, st);
  block_sum<2>(sh, adj);
  const int64_t nnz = st[0], distinct = st[1], sum_c2 = st[2];
  if (a.head_stats && tid == 0) {
    int64_t* hs = a.head_stats + (int64_t)h * 6;
    hs[0] = nnz;
    hs[1] = distinct;
    hs[2] = adj[0];
    hs[3] = adj[1];
    hs[4] = sum_c2;
    hs[5] = 0;
  }
  if (a.stats_only) return {HEAD_DONE, 0, nnz, sum_c2, adj[0], adj[1]};

  // ---- phase 1: skip cases 1-3 ----
  if (tid == 0) {
    int f = 0;
    const double kvb = (double)(2 * a.block * a.head_dim * 2);
    if ((double)distinct * kvb <= a.prof.cache_bytes) f |= FLAG_FITS_CACHE;
    const double saving = (double)nnz * a.prof.gain_ns_per_block;
    // the cost curve of the form that builds this head: one workgroup for small heads, else sliced
    const bool fused = (double)m <= a.prof.fused_max_blocks;
    const double c0 = fused ? a.prof.ovh_fused_ns_fixed : a.prof.ovh_ns_fixed;
    const double c1 = fused ? a.prof.ovh_fused_ns_per_row : a.prof.ovh_ns_per_row;
    const double c2 = fused ? a.prof.ovh_fused_ns_per_nnz : a.prof.ovh_ns_per_nnz;
    const double cost = c0 + c1 * (double)m + c2 * (double)nnz;
    if (saving < cost) f |= FLAG_LITTLE_WORK;
    if (adj[1] > 0 && (double)adj[0] / (double)adj[1] >= a.prof.j_max) f |= FLAG_LOCAL;
    sh.i32[1] = f;
  }
  __syncthreads();
  const int flags = sh.i32[1];
  PermState* S = a.state + h;
  if (a.skip_mode == SKIP_ALWAYS || (a.skip_mode == SKIP_AUTO && flags != 0)) {
    write_identity(a, sh, h, flags, true);
    if (tid == 0) {
      S->maxy = 0;
      S->active = 0;
      S->degen = 0;
      S->done = 1;
      S->flags = flags;
    }
    return {HEAD_DONE, flags, nnz, sum_c2, adj[0], adj[1]};
  }

  // ---- phase 2 starts: seeded start block and its QR ----
  int64_t zr[PER][2];
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int i = tid + k * NT;
    const uint64_t base = a.seed + 2ull * ((uint64_t)h * (uint64_t)m + (uint64_t)i);
    zr[k][0] = i < m ? (int64_t)(splitmix64(base) >> 40) - (1ll << 23) : 0;
    zr[k][1] = i < m ? (int64_t)(splitmix64(base + 1ull) >> 40) - (1ll << 23) : 0;
  }
  const bool degen = orth(sh, H, zr);
  if (!degen) store_x(a, sh, h);
  if (tid == 0) {
    S->maxy = 0;
    S->active = degen ? 0 : 1;
    S->degen = degen ? 1 : 0;
    S->done = 0;
    S->flags = flags;
    S->nnz = nnz;
    S->sum_c2 = sum_c2;
    S->adj_and = adj[0];
    S->adj_or = adj[1];
  }
  return {degen ? HEAD_DEGENERATE : HEAD_ITERATE, flags, nnz, sum_c2, adj[0], adj[1]};
}

__global__ __launch_bounds__(NT) void perm_init_kernel(WaPermLaunch a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem_raw[];
  Shared& sh = *reinterpret_cast<Shared*>(smem_raw);
  init_head(a, sh, blockIdx.x);
}

// One QR of the subspace iteration: Z from the partial sums, Cholesky-QR into the next X.
__global__ __launch_bounds__(NT) void orth_step_kernel(WaPermLaunch a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem_raw[];
  Shared& sh = *reinterpret_cast<Shared*>(smem_raw);
  const int h = blockIdx.x;
  PermState* S = a.state + h;
  if (!S->active) return;
  const Head H = head_of(a, h);
  int64_t zr[PER][2];
  load_z(a, h, zr);
  const bool degen = orth(sh, H, zr);
  if (!degen) store_x(a, sh, h);
  if (threadIdx.x == 0) {
    S->maxy = 0;
    if (degen) {
      S->active = 0;
      S->degen = 1;
    }
  }
}

// Rayleigh-Ritz on the last product Z (thread-owned rows, zr) of X (in sh.xs), canonical sign, skip
// case 4, Stage 1 and Stage 2, then case 3 against the built order. maxy is the max |Ym| of that
// product's first half (it fixes sy); adj_and / adj_or: the natural order's adjacent-row overlap.
__device__ void finish_head(const WaPermLaunch& a, Shared& sh, int h, bool degen, int64_t nnz, int64_t sum_c2,
                            int flags, uint64_t maxy, const int64_t (&zr)[PER][2], int64_t adj_and,
                            int64_t adj_or) {
  const int tid = threadIdx.x;
  const int m = a.m;
  const Head H = head_of(a, h);
  int32_t* perm = a.perm + (int64_t)h * m;
  int32_t* seg_out = a.seg_start ? a.seg_start + (int64_t)h * (a.n_xcd + 1) : nullptr;
  int64_t trace = 0;
  int scale_exp = 0;
  if (!degen) {
    const int bly = bitlen_u64(maxy);
    const int sy = bly > 30 ? bly - 30 : 0;
    uint64_t mx = 0;
#pragma unroll
    for (int k = 0; k < PER; ++k)
      if (tid + k * NT < m) {
        const uint64_t p = uabs64(zr[k][0]), q = uabs64(zr[k][1]);
        mx = p > mx ? p : mx;
        mx = q > mx ? q : mx;
      }
    mx = block_max(sh, mx);  // its barriers also publish sh.xs
    const int bl = bitlen_u64(mx);
    const int s_r = bl > 24 ? bl - 24 : 0;
    int64_t b[4] = {0, 0, 0, 0};
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int i = tid + k * NT;
      if (i < m) {
        const int64_t x0 = sh.xs[2 * i] >> 6, x1 = sh.xs[2 * i + 1] >> 6;
        const int64_t z0 = zr[k][0] >> s_r, z1 = zr[k][1] >> s_r;
        b[0] += x0 * z0;
        b[1] += x0 * z1;
        b[2] += x1 * z0;
        b[3] += x1 * z1;
      }
    }
    block_sum<4>(sh, b);
    trace = b[0] + b[3];
    scale_exp = sy + s_r + 6 - 60;
    if (tid == 0) {
      const double A = (double)b[0], C = (double)b[3], B = (double)((b[1] + b[2]) >> 1);
      double t = 0.0, cs = 1.0, sn = 0.0;
      if (B != 0.0) {
        const double tau = (C - A) / (2.0 * B);
        const double sgn = tau >= 0.0 ? 1.0 : -1.0;
        t = sgn / (__builtin_fabs(tau) + __builtin_sqrt(1.0 + tau * tau));
        cs = 1.0 / __builtin_sqrt(1.0 + t * t);
        sn = t * cs;
      }
      const double lam0 = A - t * B, lam1 = C + t * B;
      sh.dbl[3] = cs;
      sh.dbl[4] = sn;
      sh.i32[2] = lam1 > lam0 ? 1 : 0;
    }
    __syncthreads();
    const double cs = sh.dbl[3], sn = sh.dbl[4];
    const bool swp = sh.i32[2] != 0;
    for (int i = tid; i < m; i += NT) {
      const double x0 = (double)sh.xs[2 * i], x1 = (double)sh.xs[2 * i + 1];
      const int32_t u0 = (int32_t)__builtin_rint(cs * x0 - sn * x1);
      const int32_t u1 = (int32_t)__builtin_rint(sn * x0 + cs * x1);
      sh.xs[2 * i] = swp ? u1 : u0;
      sh.xs[2 * i + 1] = swp ? u0 : u1;
    }
    __syncthreads();
    // canonical sign: the entry of largest magnitude (smallest row on ties) is positive
    for (int k = 0; k < 2; ++k) {
      uint64_t key = 0;
      for (int i = tid; i < m; i += NT) {
        const uint64_t c = ((uint64_t)uabs64(sh.xs[2 * i + k]) << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)i);
        key = c > key ? c : key;
      }
      key = block_max(sh, key);
      const int istar = (int)(0xFFFFFFFFu - (uint32_t)(key & 0xFFFFFFFFull));
      const bool neg = sh.xs[2 * istar + k] < 0;
      __syncthreads();
      if (neg)
        for (int i = tid; i < m; i += NT) sh.xs[2 * i + k] = -sh.xs[2 * i + k];
      __syncthreads();
    }
  }

  // ---- phase 3: skip case 4 ----
  if (tid == 0) {
    int f = flags;
    if (degen) {
      f |= FLAG_DEGENERATE;
    } else {
      const double den = (double)m * (double)((int64_t)m * nnz - sum_c2);
      const double eta = den <= 0.0 ? 0.0 : __builtin_ldexp((double)trace, scale_exp) / den;
      if (eta < a.prof.eta_min) f |= FLAG_UNSTRUCTURED;
    }
    sh.i32[1] = f;
  }
  __syncthreads();
  flags = sh.i32[1];
  if (a.embedding)
    for (int i = tid; i < m; i += NT) {
      a.embedding[((int64_t)h * m + i) * 2] = degen ? 0 : sh.xs[2 * i];
      a.embedding[((int64_t)h * m + i) * 2 + 1] = degen ? 0 : sh.xs[2 * i + 1];
    }
  if (a.skip_mode == SKIP_AUTO && (flags & FLAG_UNSTRUCTURED)) {
    __syncthreads();  // every thread has written its embedding rows (read from sh.xs)
    write_identity(a, sh, h, flags, false);
    return;
  }

  // ---- phase 4: Stage 1, exact polar-angle order ----
  int P = 1;
  while (P < m) P <<= 1;
  int32_t* idx = sh.ys;
  if (m <= kRankSortMax) {
    // rank sort: a row's position is the number of rows that precede it (a total order)
    const int t = lanes_per_line(m);
    const int line = tid / t, sub = tid % t;
    int64_t r = 0;
    if (line < m && !degen)
      for (int j = sub; j < m; j += t) r += angle_less(sh, j, line) ? 1 : 0;
    r = group_sum(r, t);
    if (line < m && sub == 0) idx[degen ? line : (int)r] = line;  // degenerate: the identity
    __syncthreads();
    for (int i = tid; i < m; i += NT) sh.cc[i] = idx[i];
  } else if (degen) {
    for (int i = tid; i < m; i += NT) sh.cc[i] = i;
  } else {
    // bitonic sort of (x, y, row) entries, which span sh.xs and sh.ys (U is not needed after this
    // phase): each compare reads its two entries with one 16-byte load each; padding entries
    // (row -1) order last
    int32_t ux[PER], uy[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int i = tid + k * NT;
      ux[k] = i < m ? sh.xs[2 * i] : 0;
      uy[k] = i < m ? sh.xs[2 * i + 1] : 0;
    }
    __syncthreads();
    int4* ent = reinterpret_cast<int4*>(sh.xs);
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int i = tid + k * NT;
      if (i < P) ent[i] = i < m ? make_int4(ux[k], uy[k], i, 0) : make_int4(0, 0, -1, 0);
    }
    __syncthreads();
    for (int k = 2; k <= P; k <<= 1)
      for (int j = k >> 1; j > 0; j >>= 1) {
        for (int t = tid; t < P / 2; t += NT) {
          const int i = (t / j) * 2 * j + (t % j);
          const int p = i + j;
          const int4 x = ent[i], y = ent[p];
          const bool up = (i & k) == 0;
          if (up ? entry_less(y, x) : entry_less(x, y)) {
            ent[i] = y;
            ent[p] = x;
          }
        }
        __syncthreads();
      }
    for (int i = tid; i < m; i += NT) sh.cc[i] = ent[i].z;
  }
  __syncthreads();
  if (a.stage1)
    for (int i = tid; i < m; i += NT) a.stage1[(int64_t)h * m + i] = sh.cc[i];

  // ---- phase 5: work-balanced segments, wave buckets, Stage 2 ----
  compute_segments(sh, H.row_nnz, m, a.n_xcd, seg_out);
  int32_t* segof = sh.xs;  // segment of each position, left by compute_segments
  uint64_t* keys = reinterpret_cast<uint64_t*>(sh.ys);
  for (int p = tid; p < P; p += NT) {
    if (p >= m) {
      keys[p] = ~0ull;
      continue;
    }
    const int x = segof[p];
    const int off = p - sh.seg[x];
    const uint64_t bucket = ((uint64_t)x << 12) | (uint64_t)(off / a.wave);
    const int row = sh.cc[p];
    const uint64_t nz = (uint64_t)H.row_nnz[row];
    keys[p] = (bucket << 32) | ((0xFFFFull - nz) << 16) | (uint64_t)p;
  }
  __syncthreads();
  int32_t* fin = sh.xs;  // the built order (the segment map is no longer needed)
  if (m <= kRankSortMax) {
    // rank sort of the (distinct) keys
    const int t = lanes_per_line(m);
    const int line = tid / t, sub = tid % t;
    int64_t r = 0;
    if (line < m) {
      const uint64_t kp = keys[line];
      for (int q = sub; q < m; q += t) r += keys[q] < kp ? 1 : 0;
    }
    r = group_sum(r, t);
    __syncthreads();  // every key is read before the order overwrites the segment map
    if (line < m && sub == 0) fin[(int)r] = sh.cc[line];
  } else {
    for (int k = 2; k <= P; k <<= 1)
      for (int j = k >> 1; j > 0; j >>= 1) {
        for (int t = tid; t < P / 2; t += NT) {
          const int i = (t / j) * 2 * j + (t % j);
          const int p = i + j;
          const uint64_t x = keys[i], y = keys[p];
          const bool up = (i & k) == 0;
          if (up ? (y < x) : (x < y)) {
            keys[i] = y;
            keys[p] = x;
          }
        }
        __syncthreads();
      }
    for (int s = tid; s < m; s += NT) fin[s] = sh.cc[(int)(keys[s] & 0xFFFFull)];
  }
  __syncthreads();
  for (int s = tid; s < m; s += NT) perm[s] = fin[s];

  // ---- case 3 against the built order: it must raise the adjacent-row overlap ----
  if (a.skip_mode == SKIP_AUTO) {
    int64_t ov[2] = {0, 0};
    for (int t = tid; t < (m - 1) * H.nw; t += NT) {
      const int w = t / (m - 1), s = t % (m - 1);
      const uint64_t x = H.rowbits[(int64_t)w * m + fin[s]], y = H.rowbits[(int64_t)w * m + fin[s + 1]];
      ov[0] += __popcll(x & y);
      ov[1] += __popcll(x | y);
    }
    block_sum<2>(sh, ov);
    if (ov[0] * adj_or <= adj_and * ov[1]) {  // J(built order) <= J(natural order), exactly
      write_identity(a, sh, h, flags | FLAG_LOCAL, false);
      return;
    }
  }
  if (a.flags && tid == 0) a.flags[h] = (uint8_t)flags;
}

__global__ __launch_bounds__(NT) void perm_finish_kernel(WaPermLaunch a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem_raw[];
  Shared& sh = *reinterpret_cast<Shared*>(smem_raw);
  const int h = blockIdx.x;
  const PermState* S = a.state + h;
  if (S->done) return;
  const bool degen = S->degen != 0;
  int64_t zr[PER][2] = {};
  if (!degen) {
    const int2* xg = reinterpret_cast<const int2*>(a.xg) + (int64_t)h * a.m;
    for (int i = threadIdx.x; i < a.m; i += NT) {
      const int2 x = xg[i];
      sh.xs[2 * i] = x.x;
      sh.xs[2 * i + 1] = x.y;
    }
    load_z(a, h, zr);
  }
  finish_head(a, sh, h, degen, S->nnz, S->sum_c2, S->flags, S->maxy, zr, S->adj_and, S->adj_or);
}

// ---------------------------------------------------------------------------------------------
// The whole permutation of a head in one workgroup, with both centred products on the matrix cores.
//
// An integer v with |v| <= 2^31 - 2^25 is the sum of its four balanced base-256 digits,
// v = sum_b d_b 256^b with d_b in [-128, 127] (d_0 is the low byte read as a signed byte, then
// v <- (v - d_0) / 256, exactly, and so on; the last digit stays in range because the lower ones add
// at most 128 (1 + 256 + 65536) < 2^23 to it). X (2^30 per unit, a column of an orthonormal block) and
// Ys (30 significant bits) stay within 2^30 + 1. So M^T X = sum_b 256^b (M^T D_b), where D_b holds digit
// b of every entry of X: each term is a product of a 0/1 matrix and an int8 matrix, whose int32
// sums are exact (at most 1024 * 128 in magnitude), and the terms are combined exactly in int64.
// One v_mfma_i32_16x16x64_i8 takes 64 rows of 16 columns of M: A = the eight digit rows (two
// columns of X, four digits each; rows 8-15 zero), B = the 16 columns' bits. Lane l supplies bits
// [16 (l / 16), +16) of the 64-bit word of line 16 t + l mod 16, expanded to one byte per bit, and
// the digits of the same 16 rows; it receives digit rows 4 (l / 16) .. +3 of that line, so lanes
// 0-15 hold the line's product with the first column of X and lanes 16-31 with the second. M Ys
// reads the row words the same way. The products are the same integers as the sparse sums of the
// sliced form, so the result is the same bit for bit; what this form removes is the latency of the
// sparse walks and their LDS atomics.
constexpr int kMfmaMax = NT;  // rows and columns of the heads built in this form: one row or column a thread
typedef int v4i __attribute__((ext_vector_type(4)));

struct MfmaLds {
  int8_t xd[8][kMfmaMax];    // digit rows of X: row 4 k + b holds digit b of column k (zero past m)
  int8_t yd[8][kMfmaMax];    // the same for Ys (zero past n)
  int64_t v[2 * kMfmaMax];   // Ym of the first product, then Z of the second: [line][column of X]
  int32_t cc[kMfmaMax];      // column counts
  int64_t red[2][4][NWAVE];  // wavefront partials of the reductions, two alternating slot sets
};
constexpr size_t kMfmaLdsOffset = (sizeof(Shared) + 15) & ~(size_t)15;

// 16 bits -> 16 bytes of 0 or 1: byte t = bit t (each nibble spread by one 24-bit multiply)
__device__ __forceinline__ v4i bits_to_bytes(uint32_t b) {
  v4i r;
  r[0] = (int)(((b & 0xFu) * 0x204081u) & 0x01010101u);
  r[1] = (int)((((b >> 4) & 0xFu) * 0x204081u) & 0x01010101u);
  r[2] = (int)((((b >> 8) & 0xFu) * 0x204081u) & 0x01010101u);
  r[3] = (int)((((b >> 12) & 0xFu) * 0x204081u) & 0x01010101u);
  return r;
}

// Balanced base-256 digits of v into digit rows row0 .. row0 + 3, column idx.
template <int STRIDE>
__device__ __forceinline__ void put_digits(int8_t (*d)[STRIDE], int row0, int idx, int32_t v) {
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const int8_t db = (int8_t)(uint8_t)(uint32_t)v;
    d[row0 + b][idx] = db;
    v = (v - (int32_t)db) >> 8;  // exact: v - db is a multiple of 256
  }
}

// Scheduling fence between the phases of the matrix-core form: no instruction moves across it. Left
// alone, the compiler interleaves the phases (the products, the reductions, the fp64 Cholesky factor)
// in a way that made the kernel three times slower than the same code with these fences.
#define WA_PHASE_FENCE() __builtin_amdgcn_sched_barrier(0)

// Sum over the 16 lanes of each DPP row (quad exchanges, then the half-row and row mirrors); every
// lane of the row receives the row's total.
__device__ __forceinline__ int64_t row16_sum(int64_t v) {
  uint64_t u = (uint64_t)v;
  u += dpp64<0xB1, 0xf>(u);   // quad_perm [1,0,3,2]
  u += dpp64<0x4E, 0xf>(u);   // quad_perm [2,3,0,1]
  u += dpp64<0x141, 0xf>(u);  // row_half_mirror
  u += dpp64<0x140, 0xf>(u);  // row_mirror
  return (int64_t)u;
}
__device__ __forceinline__ uint64_t row16_max(uint64_t v) {
  v = max64(v, dpp64<0xB1, 0xf>(v));
  v = max64(v, dpp64<0x4E, 0xf>(v));
  v = max64(v, dpp64<0x141, 0xf>(v));
  v = max64(v, dpp64<0x140, 0xf>(v));
  return v;
}

// Exact int64 sums of K values (or the maximum of one) over the workgroup, returned to every thread:
// each wavefront reduces its lanes, parks its partial in LDS, and after the barrier lanes 0-15 of
// every wavefront read the NWAVE partials (one read each) and reduce them within their DPP row.
// Consecutive reductions alternate between the two slot sets (buf), so a wavefront that writes the
// partials of the next reduction never overwrites ones that another is still reading. One barrier,
// which also publishes every LDS write made before the call.
static_assert(NWAVE == 16, "the partials are reduced within one 16-lane DPP row");
template <int K>
__device__ __forceinline__ void wg_sum(int64_t (*red)[4][NWAVE], int buf, int64_t (&v)[K]) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  WA_PHASE_FENCE();
#pragma unroll
  for (int k = 0; k < K; ++k) v[k] = wave_sum(v[k]);
  if (lane == 0)
#pragma unroll
    for (int k = 0; k < K; ++k) red[buf][k][w] = v[k];
  __syncthreads();
#pragma unroll
  for (int k = 0; k < K; ++k) {
    const int64_t p = lane < NWAVE ? red[buf][k][lane] : 0;
    const int64_t t = row16_sum(p);
    v[k] = (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)((uint64_t)t >> 32), 0) << 32) |
                     (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(uint64_t)t, 0));
  }
  WA_PHASE_FENCE();
}
__device__ __forceinline__ uint64_t wg_max(int64_t (*red)[4][NWAVE], int buf, uint64_t v) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  WA_PHASE_FENCE();
  v = wave_max(v);
  if (lane == 0) red[buf][0][w] = (int64_t)v;
  __syncthreads();
  const uint64_t t = row16_max(lane < NWAVE ? (uint64_t)red[buf][0][lane] : 0ull);
  const uint64_t r = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(t >> 32), 0) << 32) |
                     (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)t, 0);
  WA_PHASE_FENCE();
  return r;
}

// Exact products of the digit rows dg with the bitmask of `lines` lines (word s of line j at
// bits16[4 (s lines + j) .. +3], `words` words a line). Wavefront w of the WAVES in the workgroup takes
// the 16-line tiles t0 + w, t0 + w + WAVES, ... below t1; for each, f(line, column, value) is called in
// lanes 0-31 with the product of line 16 t + l mod 16 with column l / 16 of the digit block (line may
// lie past `lines`). The bits of CH words are loaded together. With PIPE the wavefront walks its
// (tile, chunk of CH words) steps in order and loads the bits of the next step while it multiplies the
// current one, so that load latency overlaps the work (the product kernels of the sliced form, whose
// workgroups are short-lived); without, each chunk's loads are waited for before its products (the
// one-workgroup form, whose sixteen wavefronts hide each other's latency and which has no registers to
// spare: the pipelined walk there measured 1-6% slower).
template <int STRIDE, int WAVES, int CH, bool PIPE, typename F>
__device__ __forceinline__ void mfma_product(const int8_t (*dg)[STRIDE], const uint16_t* bits16, int lines,
                                             int words, int t0, int t1, F&& f) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int r = lane & 15, q = lane >> 4;
  const v4i zero = {0, 0, 0, 0};
  const int tend = min(t1, (lines + 15) >> 4);
  const int chunks = (words + CH - 1) / CH;
  // A line past the head reads the head's last line instead: its products land in output columns the
  // callers never read. Likewise A rows 8-15 repeat the digit rows: their products land in lanes 32-63.
  auto load = [&](int tile, int c, uint32_t (&bt)[CH]) {
    const int line = min(16 * tile + r, lines - 1);
#pragma unroll
    for (int u = 0; u < CH; ++u) {
      const int s = c * CH + u;
      bt[u] = s < words ? bits16[(s * lines + line) * 4 + q] : 0u;
    }
  };
  WA_PHASE_FENCE();
  if constexpr (!PIPE) {
    for (int tile = t0 + w; tile < tend; tile += WAVES) {
      v4i acc = zero;
      for (int c = 0; c < chunks; ++c) {
        uint32_t bt[CH];
        load(tile, c, bt);
#pragma unroll
        for (int u = 0; u < CH; ++u) {
          const int s = c * CH + u;
          if (s < words) {
            const v4i av = *(const v4i*)&dg[r & 7][64 * s + 16 * q];
            acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(av, bits_to_bytes(bt[u]), acc, 0, 0, 0);
          }
        }
      }
      if (q < 2) f(16 * tile + r, q, (int64_t)acc[0] + 256ll * acc[1] + 65536ll * acc[2] + 16777216ll * acc[3]);
    }
    WA_PHASE_FENCE();
    return;
  }
  int tile = t0 + w, c = 0;
  if (tile < tend) {
    uint32_t cur[CH], nxt[CH];
    load(tile, 0, cur);
    v4i acc = zero;
    for (;;) {
      // the step after (tile, c)
      int ntile = tile, nc = c + 1;
      if (nc == chunks) {
        ntile = tile + WAVES;
        nc = 0;
      }
      if (ntile < tend) load(ntile, nc, nxt);
#pragma unroll
      for (int u = 0; u < CH; ++u) {
        const int s = c * CH + u;
        if (s < words) {
          const v4i av = *(const v4i*)&dg[r & 7][64 * s + 16 * q];
          acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(av, bits_to_bytes(cur[u]), acc, 0, 0, 0);
        }
      }
      if (nc == 0) {  // the tile is complete
        if (q < 2) f(16 * tile + r, q, (int64_t)acc[0] + 256ll * acc[1] + 65536ll * acc[2] + 16777216ll * acc[3]);
        acc = zero;
      }
      if (ntile >= tend) break;
      tile = ntile;
      c = nc;
#pragma unroll
      for (int u = 0; u < CH; ++u) cur[u] = nxt[u];
    }
  }
  WA_PHASE_FENCE();
}

__global__ __launch_bounds__(NT) void perm_mfma_kernel(WaPermLaunch a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem_raw[];
  Shared& sh = *reinterpret_cast<Shared*>(smem_raw);
  MfmaLds& L = *reinterpret_cast<MfmaLds*>(smem_raw + kMfmaLdsOffset);
  const int h = blockIdx.x;
  const HeadInit hi = init_head(a, sh, h);
  if (hi.status == HEAD_DONE) return;
  bool degen = hi.status == HEAD_DEGENERATE;
  int64_t zr[PER][2] = {};
  uint64_t maxy = 0;
  if (!degen) {
    const int tid = threadIdx.x;  // row tid (QR) and column tid (Ys) of the head
    const int m = a.m, n = a.n;
    const int64_t mm = m;
    const Head H = head_of(a, h);
    const uint16_t* cb16 = reinterpret_cast<const uint16_t*>(H.colbits);
    const uint16_t* rb16 = reinterpret_cast<const uint16_t*>(H.rowbits);
    // digit rows start at zero (their padding past m and n stays zero); X of the seeded start
    for (int e = tid; e < 8 * kMfmaMax / 4; e += NT) {
      reinterpret_cast<int32_t*>(L.xd)[e] = 0;
      reinterpret_cast<int32_t*>(L.yd)[e] = 0;
    }
    L.cc[tid] = tid < n ? a.cc[(int64_t)h * n + tid] : 0;
    __syncthreads();
    int64_t sx[2] = {0, 0};  // 1^T X
    if (tid < m) {
      const int32_t x0 = sh.xs[2 * tid], x1 = sh.xs[2 * tid + 1];
      put_digits(L.xd, 0, tid, x0);
      put_digits(L.xd, 4, tid, x1);
      sx[0] = x0;
      sx[1] = x1;
    }
    int rb = 0;                      // reductions so far (selects the slot set)
    wg_sum<2>(L.red, rb++ & 1, sx);  // its barrier also publishes the digits
    for (int it = 0; it <= a.iters; ++it) {
      // ---- Ym = m M^T X - c (1^T X), and max |Ym| ----
      uint64_t mx = 0;
      mfma_product<kMfmaMax, NWAVE, 4, false>(L.xd, cb16, n, H.mw, 0, kMfmaMax / 16, [&](int j, int k, int64_t ya) {
        if (j < n) {
          const int64_t y = mm * ya - (int64_t)L.cc[j] * (k == 0 ? sx[0] : sx[1]);
          L.v[2 * j + k] = y;
          mx = max64(mx, uabs64(y));
        }
      });
      maxy = wg_max(L.red, rb++ & 1, mx);  // its barrier also publishes Ym
      const int bly = bitlen_u64(maxy);
      const int sy = bly > 30 ? bly - 30 : 0;
      // ---- Ys = Ym >> sy as digit rows, and c^T Ys ----
      int64_t py[2] = {0, 0};
      if (tid < n) {
        const int32_t v0 = (int32_t)(L.v[2 * tid] >> sy), v1 = (int32_t)(L.v[2 * tid + 1] >> sy);
        put_digits(L.yd, 0, tid, v0);
        put_digits(L.yd, 4, tid, v1);
        py[0] = (int64_t)L.cc[tid] * v0;
        py[1] = (int64_t)L.cc[tid] * v1;
      }
      wg_sum<2>(L.red, rb++ & 1, py);  // its barrier also publishes the Ys digits (Ym is read)
      // ---- Z = m M Ys - 1 (c^T Ys), and max |Z| ----
      uint64_t mz = 0;
      mfma_product<kMfmaMax, NWAVE, 4, false>(L.yd, rb16, m, H.nw, 0, kMfmaMax / 16, [&](int i, int k, int64_t za) {
        if (i < m) {
          const int64_t z = mm * za - (k == 0 ? py[0] : py[1]);
          L.v[2 * i + k] = z;
          mz = max64(mz, uabs64(z));
        }
      });
      mz = wg_max(L.red, rb++ & 1, mz);  // its barrier also publishes Z
      int64_t z0 = 0, z1 = 0;
      if (tid < m) {
        z0 = L.v[2 * tid];
        z1 = L.v[2 * tid + 1];
      }
      if (it == a.iters) {  // the last product: Rayleigh-Ritz in the finishing phases
        zr[0][0] = z0;
        zr[0][1] = z1;
        break;
      }
      // ---- Cholesky-QR: X = Z R^-1 ----
      const int blz = bitlen_u64(mz);
      const int s = blz > 24 ? blz - 24 : 0;
      const int64_t z0s = z0 >> s, z1s = z1 >> s;
      int64_t g[3] = {z0s * z0s, z0s * z1s, z1s * z1s};
      wg_sum<3>(L.red, rb++ & 1, g);
      if (g[0] == 0) {  // uniform: every thread holds the same sums
        degen = true;
        break;
      }
      const Chol c = chol2(g);
      sx[0] = 0;
      sx[1] = 0;
      if (tid < m) {
        int32_t x0, x1;
        orth_row(c, z0s, z1s, x0, x1);
        sh.xs[2 * tid] = x0;
        sh.xs[2 * tid + 1] = x1;
        put_digits(L.xd, 0, tid, x0);
        put_digits(L.xd, 4, tid, x1);
        sx[0] = x0;
        sx[1] = x1;
      }
      wg_sum<2>(L.red, rb++ & 1, sx);  // its barrier also publishes X and its digits
    }
  }
  finish_head(a, sh, h, degen, hi.nnz, hi.sum_c2, hi.flags, maxy, zr, hi.adj_and, hi.adj_or);
}

// ---------------------------------------------------------------------------------------------
// Centred products across many workgroups, for heads of more than kMfmaMax blocks. One subspace step
// X -> Z = m * M~ Ys, with Ys = (m * M~^T X) >> sy, runs as two product kernels and the per-head orth
// kernel. A product workgroup (GT threads) takes kSliceTiles consecutive 16-line tiles of one head, dealt
// to its wavefronts in turn, and computes them with the matrix-core products of perm_mfma_kernel over
// the whole head:
//   gather:  the digit rows of X and 1^T X (each workgroup of the head builds them in LDS), then
//            Ym[j] = m * (M^T X)[j] - c_j * 1^T X for its columns, and an atomic max of |Ym| per head;
//   scatter: the digit rows of Ys = Ym >> sy and c^T Ys (likewise), then Z[i] = m * (M Ys)[i] - c^T Ys
//            for its rows;
//   orth:    the Cholesky-QR of Z, the next X.
// Every workgroup of a head computes the same exact sums and each line is written by one lane, so the
// slicing does not change any result.
constexpr int GT = 256;
constexpr int GW = GT / 64;
constexpr int kSliceTiles = 8;  // 16-line tiles per product workgroup (two per wavefront)
constexpr int kLoadBatch = 8;   // X rows or Ym columns per thread whose loads are issued together

struct SliceLds {
  int8_t dg[8][MAXB];  // digit rows of X (gather) or Ys (scatter), zero past the head's last word
  int64_t red[GW][2];
};

// Exact sums of two int64 values over a GT-thread workgroup, returned to every thread; its barrier
// also publishes every LDS write made before the call.
__device__ __forceinline__ void slice_sum2(int64_t (*red)[2], int64_t& v0, int64_t& v1) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  v0 = wave_sum(v0);
  v1 = wave_sum(v1);
  if (lane == 0) {
    red[w][0] = v0;
    red[w][1] = v1;
  }
  __syncthreads();
  v0 = 0;
  v1 = 0;
#pragma unroll
  for (int k = 0; k < GW; ++k) {
    v0 += red[k][0];
    v1 += red[k][1];
  }
}

__global__ __launch_bounds__(GT) void mfma_gather_kernel(WaPermLaunch a) {
  const int h = blockIdx.x / a.slices, g = blockIdx.x % a.slices;
  if (!a.state[h].active) return;
  __shared__ __attribute__((aligned(16))) SliceLds L;
  __shared__ uint64_t redm[GW];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int m = a.m, n = a.n;
  const Head H = head_of(a, h);
  const int2* xg = reinterpret_cast<const int2*>(a.xg) + (int64_t)h * m;
  int64_t sx0 = 0, sx1 = 0;
  for (int i0 = 0; i0 < 64 * H.mw; i0 += kLoadBatch * GT) {  // the rows' loads in flight together
    int2 x[kLoadBatch];
#pragma unroll
    for (int u = 0; u < kLoadBatch; ++u) {
      const int i = i0 + u * GT + tid;
      x[u] = i < m ? xg[i] : make_int2(0, 0);
    }
#pragma unroll
    for (int u = 0; u < kLoadBatch; ++u) {
      const int i = i0 + u * GT + tid;
      if (i < 64 * H.mw) {
        put_digits(L.dg, 0, i, x[u].x);
        put_digits(L.dg, 4, i, x[u].y);
        sx0 += x[u].x;
        sx1 += x[u].y;
      }
    }
  }
  slice_sum2(L.red, sx0, sx1);  // its barrier also publishes the digits
  const int32_t* cc = a.cc + (int64_t)h * n;
  int64_t* ym = a.ym + (int64_t)h * n * 2;
  uint64_t mx = 0;
  mfma_product<MAXB, GW, 16, true>(L.dg, reinterpret_cast<const uint16_t*>(H.colbits), n, H.mw, g * kSliceTiles,
                             g * kSliceTiles + kSliceTiles,
                         [&](int j, int k, int64_t ya) {
                           if (j < n) {
                             const int64_t y = (int64_t)m * ya - (int64_t)cc[j] * (k == 0 ? sx0 : sx1);
                             ym[2 * j + k] = y;
                             mx = max64(mx, uabs64(y));
                           }
                         });
  mx = wave_max(mx);
  if (lane == 0) redm[w] = mx;
  __syncthreads();
  if (tid == 0) {
    for (int k = 1; k < GW; ++k) mx = max64(mx, redm[k]);
    if (mx) atomicMax((unsigned long long*)&a.state[h].maxy, (unsigned long long)mx);
  }
}

__global__ __launch_bounds__(GT) void mfma_scatter_kernel(WaPermLaunch a) {
  const int h = blockIdx.x / a.slices, g = blockIdx.x % a.slices;
  if (!a.state[h].active) return;
  __shared__ __attribute__((aligned(16))) SliceLds L;
  const int tid = threadIdx.x;
  const int m = a.m, n = a.n;
  const Head H = head_of(a, h);
  const int bl = bitlen_u64(a.state[h].maxy);
  const int sy = bl > 30 ? bl - 30 : 0;
  const int32_t* cc = a.cc + (int64_t)h * n;
  const int64_t* ym = a.ym + (int64_t)h * n * 2;
  int64_t p0 = 0, p1 = 0;  // c^T Ys
  for (int j0 = 0; j0 < 64 * H.nw; j0 += kLoadBatch * GT) {  // the columns' loads in flight together
    int64_t y0[kLoadBatch], y1[kLoadBatch];
    int32_t c[kLoadBatch];
#pragma unroll
    for (int u = 0; u < kLoadBatch; ++u) {
      const int j = j0 + u * GT + tid;
      y0[u] = j < n ? ym[2 * j] : 0;
      y1[u] = j < n ? ym[2 * j + 1] : 0;
      c[u] = j < n ? cc[j] : 0;
    }
#pragma unroll
    for (int u = 0; u < kLoadBatch; ++u) {
      const int j = j0 + u * GT + tid;
      if (j < 64 * H.nw) {
        const int32_t v0 = (int32_t)(y0[u] >> sy), v1 = (int32_t)(y1[u] >> sy);
        p0 += (int64_t)c[u] * v0;
        p1 += (int64_t)c[u] * v1;
        put_digits(L.dg, 0, j, v0);
        put_digits(L.dg, 4, j, v1);
      }
    }
  }
  slice_sum2(L.red, p0, p1);  // its barrier also publishes the digits
  int64_t* z = a.z + (int64_t)h * m * 2;
  mfma_product<MAXB, GW, 16, true>(L.dg, reinterpret_cast<const uint16_t*>(H.rowbits), m, H.nw, g * kSliceTiles,
                             g * kSliceTiles + kSliceTiles,
                         [&](int i, int k, int64_t za) {
                           if (i < m) z[2 * i + k] = (int64_t)m * za - (k == 0 ? p0 : p1);
                         });
}

// Arithmetic self-check: the fp64 operations the permutation relies on, evaluated on the GPU.
__global__ void fp64_probe_kernel(const double* a, const double* b, const int64_t* c, double* out, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const double x = a[i], y = b[i];
  out[6 * i + 0] = __builtin_sqrt(__builtin_fabs(x));
  out[6 * i + 1] = x / y;
  out[6 * i + 2] = (double)c[i];
  out[6 * i + 3] = __builtin_rint(x * 1073741824.0);
  out[6 * i + 4] = x * y - y * 3.0;
  out[6 * i + 5] = __builtin_ldexp(x, (int)(c[i] & 31) - 16);
}

}  // namespace

size_t wa_perm_shared_bytes() { return sizeof(Shared); }

int wa_perm_slices(int n) { return (n + 16 * kSliceTiles - 1) / (16 * kSliceTiles); }

// Heads of at most this many rows and columns are built by perm_mfma_kernel (one launch, one workgroup
// a head); larger ones by the slice kernels (3 + 3 T launches), whose column slices spread a head over
// the whole chip.
constexpr int kMfmaFormMax = kMfmaMax;
static_assert(kMfmaLdsOffset + sizeof(MfmaLds) <= 160 * 1024, "the matrix-core form fits one workgroup's LDS");

// Launch sequence on one stream: the matrix-core kernel alone; or init, iters x (gather, scatter,
// orth), gather, scatter, finish. The statistics-only form runs init alone.
hipError_t wa_launch_perm(const WaPermLaunch& a, hipStream_t stream) {
  if (a.bh <= 0) return hipSuccess;
  if (a.slices != wa_perm_slices(a.m > a.n ? a.m : a.n) || a.m > MAXB || a.n > MAXB) return hipErrorInvalidValue;
  const size_t smem = sizeof(Shared);
  const void* big[] = {(const void*)perm_init_kernel, (const void*)orth_step_kernel, (const void*)perm_finish_kernel};
  hipError_t e;
  for (const void* f : big)
    if ((e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem)) != hipSuccess) return e;
  const size_t msmem = kMfmaLdsOffset + sizeof(MfmaLds);
  if (!a.stats_only && a.m <= kMfmaFormMax && a.n <= kMfmaFormMax) {
    e = hipFuncSetAttribute((const void*)perm_mfma_kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)msmem);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(perm_mfma_kernel, dim3(a.bh), dim3(NT), msmem, stream, a);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(perm_init_kernel, dim3(a.bh), dim3(NT), smem, stream, a);
  if ((e = hipGetLastError()) != hipSuccess || a.stats_only) return e;
  const dim3 slices((unsigned)(a.bh * a.slices));
  for (int it = 0; it <= a.iters; ++it) {
    hipLaunchKernelGGL(mfma_gather_kernel, slices, dim3(GT), 0, stream, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(mfma_scatter_kernel, slices, dim3(GT), 0, stream, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (it < a.iters) {
      hipLaunchKernelGGL(orth_step_kernel, dim3(a.bh), dim3(NT), smem, stream, a);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
  }
  hipLaunchKernelGGL(perm_finish_kernel, dim3(a.bh), dim3(NT), smem, stream, a);
  return hipGetLastError();
}

hipError_t wa_launch_fp64_probe(const double* a, const double* b, const int64_t* c, double* out, int n,
                                hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fp64_probe_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, a, b, c, out, n);
  return hipGetLastError();
}
