// Mask scans for gfx950: row counts, per-row KV-index lists, and the bit-packed
// row and column masks that the permutation builder iterates over.
//
// A wavefront scans one mask row 1024 columns at a time: lane l takes columns
// [1024t + 16l, +16) with 16-byte loads (mask rows start at any byte, so a lane
// reads the aligned 16-byte chunk holding its first column and, when its columns
// cross into the next chunk, that one too, and byte-aligns the pair). Each load
// covers at least one byte of the row, so it never leaves the pages that hold
// the mask. Kept-column counts are popcounts; the lanes' exclusive prefix sum
// ranks their columns, so indices are written in ascending column order (the
// order in which the attention kernel visits KV blocks) and the result is
// independent of scheduling.

#include "common.h"
#include "perm_launch.h"
#include "wavealign.h"

namespace {

constexpr int kWavesPerWG = 4;

__device__ __forceinline__ uint64_t ballot64(bool p) { return __ballot(p); }

// One bit per byte of w (bit i = byte i is nonzero).
__device__ __forceinline__ uint32_t nz_nibble(uint32_t w) {
  uint32_t t = ((w & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | w;
  t = (t >> 7) & 0x01010101u;
  return (t | (t >> 7) | (t >> 14) | (t >> 21)) & 0xFu;
}

// Nonzero mask of the bytes p[0 .. valid), valid in 1..16 (bit b = byte b). The byte offset of p
// within its 16-byte chunk must be the same in every lane of the wavefront.
__device__ __forceinline__ uint32_t nz16(const uint8_t* p, int valid) {
  const uintptr_t addr = (uintptr_t)p;
  const uint8_t* a = p - (addr & 15);
  const int d = (int)(addr & 15);
  const uint4 c0 = *(const uint4*)a;
  uint4 c1 = make_uint4(0u, 0u, 0u, 0u);
  if (d + valid > 16) c1 = *(const uint4*)(a + 16);
  const uint32_t w[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
  const uint32_t r = (uint32_t)(d & 3);
  uint32_t o[4];
  switch (d >> 2) {  // uniform
    case 0:
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = __builtin_amdgcn_alignbyte(w[i + 1], w[i], r);
      break;
    case 1:
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = __builtin_amdgcn_alignbyte(w[i + 2], w[i + 1], r);
      break;
    case 2:
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = __builtin_amdgcn_alignbyte(w[i + 3], w[i + 2], r);
      break;
    default:
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = __builtin_amdgcn_alignbyte(w[i + 4], w[i + 3], r);
      break;
  }
  const uint32_t bits = nz_nibble(o[0]) | (nz_nibble(o[1]) << 4) | (nz_nibble(o[2]) << 8) | (nz_nibble(o[3]) << 12);
  return valid >= 16 ? bits : bits & ((1u << valid) - 1u);
}

// Kept-column mask of columns [col0, col0 + 16) of a row of n bytes (0 past the end).
__device__ __forceinline__ uint32_t row_bits16(const uint8_t* rowp, int n, int col0) {
  return col0 < n ? nz16(rowp + col0, min(16, n - col0)) : 0u;
}

// counts[(row / mb) * count_stride_rows + counts_offset + row % mb] = n_row
__global__ __launch_bounds__(256) void row_count_kernel(const uint8_t* __restrict__ mask, int64_t rows, int n,
                                                         int32_t* __restrict__ counts, int64_t stride, int offset,
                                                         int mb) {
  const int64_t row = (int64_t)blockIdx.x * kWavesPerWG + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int lane = threadIdx.x & 63;
  const uint8_t* p = mask + row * n;
  int cnt = 0;
  for (int c0 = 0; c0 < n; c0 += 1024) cnt += __popc(row_bits16(p, n, c0 + 16 * lane));
  for (int o = 32; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o);
  if (lane == 0) counts[(row / mb) * stride + offset + row % mb] = cnt;
}

// In place: row_ptr[h][1..mb] holds counts on entry, the exclusive scan on exit (row_ptr[h][0] = 0).
__global__ __launch_bounds__(1024) void head_scan_kernel(int32_t* __restrict__ row_ptr, int mb) {
  __shared__ int32_t part[1024];
  int32_t* rp = row_ptr + (int64_t)blockIdx.x * (mb + 1);
  const int t = threadIdx.x;
  // each thread scans a contiguous chunk
  const int per = (mb + 1023) / 1024;
  const int lo = t * per, hi = min(lo + per, mb);
  int32_t s = 0;
  for (int i = lo; i < hi; ++i) s += rp[i + 1];
  part[t] = s;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {
    int32_t v = t >= off ? part[t - off] : 0;
    __syncthreads();
    part[t] += v;
    __syncthreads();
  }
  int32_t run = t > 0 ? part[t - 1] : 0;
  for (int i = lo; i < hi; ++i) {
    const int32_t c = rp[i + 1];
    run += c;
    rp[i + 1] = run;
  }
  if (t == 0) rp[0] = 0;
}

__global__ __launch_bounds__(256) void row_write_kernel(const uint8_t* __restrict__ mask, int bh, int mb, int n,
                                                         const int32_t* __restrict__ row_ptr,
                                                         int32_t* __restrict__ col_idx) {
  const int64_t row = (int64_t)blockIdx.x * kWavesPerWG + (threadIdx.x >> 6);
  if (row >= (int64_t)bh * mb) return;
  const int lane = threadIdx.x & 63;
  const int64_t h = row / mb;
  const int i = (int)(row % mb);
  const uint8_t* p = mask + row * n;
  int32_t* out = col_idx + h * (int64_t)mb * n + row_ptr[h * (mb + 1) + i];
  int base = 0;
  for (int c0 = 0; c0 < n; c0 += 1024) {
    const int col = c0 + 16 * lane;
    uint32_t bits = row_bits16(p, n, col);
    const int cnt = __popc(bits);
    int incl = cnt;  // inclusive prefix sum over the lanes
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int u = __shfl_up(incl, o);
      if (lane >= o) incl += u;
    }
    int pos = base + incl - cnt;
    while (bits) {
      out[pos++] = col + __ffs((int)bits) - 1;
      bits &= bits - 1u;
    }
    base += __shfl(incl, 63);
  }
}

// Bit-packed rows, word-major per head: rowbits[(h*nw + w)*m + i] bit b = M[h][i][64w + b];
// row_nnz[h*m + i] = n_i.
__global__ __launch_bounds__(256) void pack_rows_kernel(const uint8_t* __restrict__ mask, int64_t rows, int m, int n,
                                                        int nw, uint64_t* __restrict__ rowbits,
                                                        int32_t* __restrict__ row_nnz) {
  const int64_t row = (int64_t)blockIdx.x * kWavesPerWG + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int lane = threadIdx.x & 63;
  const int64_t h = row / m;
  const int i = (int)(row % m);
  const uint8_t* p = mask + row * n;
  int cnt = 0;
  for (int c0 = 0; c0 < n; c0 += 1024) {
    const uint32_t b = row_bits16(p, n, c0 + 16 * lane);
    cnt += __popc(b);
    // lanes 4k .. 4k+3 hold the 64 columns of word c0 / 64 + k
    const uint64_t word = (uint64_t)b | ((uint64_t)__shfl_down(b, 1) << 16) | ((uint64_t)__shfl_down(b, 2) << 32) |
                          ((uint64_t)__shfl_down(b, 3) << 48);
    const int w = c0 / 64 + (lane >> 2);
    if ((lane & 3) == 0 && w < nw) rowbits[(h * nw + w) * m + i] = word;
  }
  for (int o = 32; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o);
  if (lane == 0) row_nnz[row] = cnt;
}

// Bit-packed columns from bit-packed rows, word-major: colbits[(h*mw + v)*n + j] bit r = M[h][64v + r][j].
// One wavefront per (head, 64-column group, 64-row group): lane r holds row 64v + r's word.
__global__ __launch_bounds__(256) void transpose_bits_kernel(const uint64_t* __restrict__ rowbits, int bh, int m,
                                                             int n, int nw, int mw,
                                                             uint64_t* __restrict__ colbits) {
  const int64_t task = (int64_t)blockIdx.x * kWavesPerWG + (threadIdx.x >> 6);
  const int64_t per_head = (int64_t)nw * mw;
  if (task >= (int64_t)bh * per_head) return;
  const int lane = threadIdx.x & 63;
  const int64_t h = task / per_head;
  const int rem = (int)(task % per_head);
  const int cw = rem / mw;   // column word
  const int v = rem % mw;    // row word
  const int r = v * 64 + lane;
  uint64_t out = r < m ? rowbits[(h * nw + cw) * m + r] : 0ull;
  // 64 x 64 bit transpose (lane = row -> lane = column) by the recursive block swap: at distance s,
  // a lane in the lower half of each 2s group trades its columns with bit s set for the partner's
  // columns with bit s clear (six lane exchanges in place of 64 ballots)
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) {
    const uint64_t lo = s == 32 ? 0x00000000FFFFFFFFull : s == 16 ? 0x0000FFFF0000FFFFull
                      : s == 8 ? 0x00FF00FF00FF00FFull : s == 4 ? 0x0F0F0F0F0F0F0F0Full
                      : s == 2 ? 0x3333333333333333ull : 0x5555555555555555ull;  // columns with bit s clear
    const uint32_t tlo = (uint32_t)__shfl_xor((int)(uint32_t)out, s);
    const uint32_t thi = (uint32_t)__shfl_xor((int)(uint32_t)(out >> 32), s);
    const uint64_t t = ((uint64_t)thi << 32) | tlo;
    out = (lane & s) ? ((out & ~lo) | ((t >> s) & lo)) : ((out & lo) | ((t & lo) << s));
  }
  const int j = cw * 64 + lane;
  if (j < n) colbits[(h * mw + v) * n + j] = out;
}

// Permutation check: one workgroup per head marks each entry in an LDS bitmap; an entry out of
// range or already marked, or a bitmap with fewer than m marks, makes the head bad. bad[0] counts
// bad heads (zeroed by the first workgroup's predecessor kernel); head_ok (nullable) gets 1 / 0.
__global__ __launch_bounds__(64) void zero_counter_kernel(int32_t* c) {
  if (threadIdx.x == 0) c[0] = 0;
}

__global__ __launch_bounds__(256) void check_perm_kernel(const int32_t* __restrict__ perm, int m,
                                                         int32_t* __restrict__ bad, int32_t* __restrict__ head_ok) {
  __shared__ uint32_t seen[WA_MAX_BLOCKS / 32];
  __shared__ int fault;
  const int64_t h = blockIdx.x;
  const int tid = threadIdx.x;
  for (int i = tid; i < (m + 31) / 32; i += 256) seen[i] = 0u;
  if (tid == 0) fault = 0;
  __syncthreads();
  const int32_t* p = perm + h * m;
  for (int s = tid; s < m; s += 256) {
    const int32_t r = p[s];
    if (r < 0 || r >= m) {
      fault = 1;
    } else {
      const uint32_t bit = 1u << (r & 31);
      if (atomicOr(&seen[r >> 5], bit) & bit) fault = 1;
    }
  }
  __syncthreads();
  if (tid == 0) {
    if (head_ok) head_ok[h] = fault ? 0 : 1;
    if (fault) atomicAdd(bad, 1);
  }
}

// Each workgroup records the XCD it runs on (hardware register XCC_ID, bits [3:0]).
__global__ void xcc_probe_kernel(int32_t* out, int n) {
  if (threadIdx.x == 0 && (int)blockIdx.x < n)
    out[blockIdx.x] = (int32_t)(__builtin_amdgcn_s_getreg((3 << 11) | (0 << 6) | 20) & 0xF);
}

}  // namespace

hipError_t wa_launch_check_perm(const int32_t* perm, int bh, int m, int32_t* bad, int32_t* head_ok,
                                hipStream_t stream) {
  hipLaunchKernelGGL(zero_counter_kernel, dim3(1), dim3(64), 0, stream, bad);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || bh <= 0) return e;
  hipLaunchKernelGGL(check_perm_kernel, dim3(bh), dim3(256), 0, stream, perm, m, bad, head_ok);
  return hipGetLastError();
}

hipError_t wa_launch_xcc_probe(int32_t* out, int n_wg, hipStream_t stream) {
  if (n_wg <= 0) return hipSuccess;
  hipLaunchKernelGGL(xcc_probe_kernel, dim3(n_wg), dim3(64), 0, stream, out, n_wg);
  return hipGetLastError();
}

hipError_t wa_launch_row_count(const uint8_t* mask, int64_t rows, int n, int32_t* counts, int64_t count_stride_rows,
                               int counts_offset, int mb, hipStream_t stream) {
  if (rows <= 0) return hipSuccess;
  const int64_t grid = (rows + kWavesPerWG - 1) / kWavesPerWG;
  hipLaunchKernelGGL(row_count_kernel, dim3((unsigned)grid), dim3(256), 0, stream, mask, rows, n, counts,
                     count_stride_rows, counts_offset, mb);
  return hipGetLastError();
}

hipError_t wa_launch_head_scan(int32_t* row_ptr, int bh, int mb, hipStream_t stream) {
  if (bh <= 0) return hipSuccess;
  hipLaunchKernelGGL(head_scan_kernel, dim3(bh), dim3(1024), 0, stream, row_ptr, mb);
  return hipGetLastError();
}

hipError_t wa_launch_row_write(const uint8_t* mask, int bh, int mb, int n, const int32_t* row_ptr, int32_t* col_idx,
                               hipStream_t stream) {
  const int64_t rows = (int64_t)bh * mb;
  if (rows <= 0) return hipSuccess;
  const int64_t grid = (rows + kWavesPerWG - 1) / kWavesPerWG;
  hipLaunchKernelGGL(row_write_kernel, dim3((unsigned)grid), dim3(256), 0, stream, mask, bh, mb, n, row_ptr, col_idx);
  return hipGetLastError();
}

hipError_t wa_launch_pack_rows(const uint8_t* mask, int64_t rows, int m, int n, uint64_t* rowbits,
                               int32_t* row_nnz, hipStream_t stream) {
  if (rows <= 0) return hipSuccess;
  const int nw = (n + 63) / 64;
  const int64_t grid = (rows + kWavesPerWG - 1) / kWavesPerWG;
  hipLaunchKernelGGL(pack_rows_kernel, dim3((unsigned)grid), dim3(256), 0, stream, mask, rows, m, n, nw, rowbits,
                     row_nnz);
  return hipGetLastError();
}

hipError_t wa_launch_transpose_bits(const uint64_t* rowbits, int bh, int m, int n, uint64_t* colbits,
                                    hipStream_t stream) {
  const int nw = (n + 63) / 64, mw = (m + 63) / 64;
  const int64_t tasks = (int64_t)bh * nw * mw;
  if (tasks <= 0) return hipSuccess;
  const int64_t grid = (tasks + kWavesPerWG - 1) / kWavesPerWG;
  hipLaunchKernelGGL(transpose_bits_kernel, dim3((unsigned)grid), dim3(256), 0, stream, rowbits, bh, m, n, nw, mw,
                     colbits);
  return hipGetLastError();
}
