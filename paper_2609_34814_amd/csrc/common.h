// Internal helpers shared by the HIP sources of the library (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// Workgroups of one head: ceil(m / n_xcd) per XCD.
__host__ __device__ inline int wg_per_xcd(int m, int n_xcd) { return (m + n_xcd - 1) / n_xcd; }
__host__ __device__ inline int wg_per_head(int m, int n_xcd) { return n_xcd * wg_per_xcd(m, n_xcd); }

// Slots [first, last) run by workgroup g of one head. Workgroups are dispatched round-robin
// over the XCDs (g mod n_xcd); the L = ceil(m / n_xcd) workgroups of XCD x run segment
// [s0, s1) of the slots in order, each taking c = ceil((s1 - s0) / L) consecutive slots.
// seg (n_xcd + 1 entries) gives the segments; without it the segments have equal row counts.
__host__ __device__ inline void xcd_slots(int g, int m, int n_xcd, const int32_t* seg, int* first, int* last) {
  const int x = g % n_xcd;
  const int l = g / n_xcd;
  const int L = wg_per_xcd(m, n_xcd);
  int s0, s1;
  if (seg) {
    s0 = min(max(seg[x], 0), m);
    s1 = min(max(seg[x + 1], s0), m);
  } else {
    const int base = m / n_xcd, extra = m % n_xcd;
    s0 = x * base + (x < extra ? x : extra);
    s1 = s0 + base + (x < extra ? 1 : 0);
  }
  const int c = (s1 - s0 + L - 1) / L;
  *first = min(s0 + l * c, s1);
  *last = min(*first + c, s1);
}

// Workgroups of one head when each workgroup runs pairs of consecutive slots.
__host__ __device__ inline int pair_wg_per_xcd(int m, int n_xcd) { return (wg_per_xcd(m, n_xcd) + 1) / 2; }
__host__ __device__ inline int pair_wg_per_head(int m, int n_xcd) { return n_xcd * pair_wg_per_xcd(m, n_xcd); }

// Slots [first, last) run, two at a time, by workgroup g of one head: the L = ceil(ceil(m/n_xcd)/2)
// workgroups of XCD x take the pairs of consecutive slots of segment x in order, c = ceil(pairs / L)
// pairs each (the last pair of a segment of odd length has one slot).
__host__ __device__ inline void xcd_pairs(int g, int m, int n_xcd, const int32_t* seg, int* first, int* last) {
  const int x = g % n_xcd;
  const int l = g / n_xcd;
  const int L = pair_wg_per_xcd(m, n_xcd);
  int s0, s1;
  if (seg) {
    s0 = min(max(seg[x], 0), m);
    s1 = min(max(seg[x + 1], s0), m);
  } else {
    const int base = m / n_xcd, extra = m % n_xcd;
    s0 = x * base + (x < extra ? x : extra);
    s1 = s0 + base + (x < extra ? 1 : 0);
  }
  const int pairs = (s1 - s0 + 1) / 2;
  const int c = (pairs + L - 1) / L;
  *first = min(s0 + 2 * l * c, s1);
  *last = min(*first + 2 * c, s1);
}

}  // namespace wa

// Launch helpers (implemented in the .hip sources, called by the ABI layer).
struct WaAttnLaunch {
  const void* q;
  const void* k;
  const void* v;
  void* vt;          // workspace: V transposed to [bh][head_dim][mb*block], zero-padded
  const int32_t* row_ptr;
  const int32_t* col_idx;
  const int32_t* perm;
  const int32_t* seg;  // [bh][n_xcd+1] XCD segment starts, nullable
  void* o;
  float* lse;
  int32_t bh;        // batch * heads
  int32_t seq_len;
  int32_t mb;        // blocks per sequence
  int32_t head_dim;
  int32_t block;
  int32_t n_xcd;
  float scale;       // softmax scale
};

hipError_t wa_launch_attention(const WaAttnLaunch& a, hipStream_t stream);
size_t wa_vt_bytes(int64_t bh, int mb, int head_dim, int block);
hipError_t wa_attention_occupancy(int head_dim, int block, int* wgs_per_cu);

hipError_t wa_launch_row_count(const uint8_t* mask, int64_t rows, int n, int32_t* counts, int64_t count_stride_rows,
                               int counts_offset, int mb, hipStream_t stream);
hipError_t wa_launch_head_scan(int32_t* row_ptr, int bh, int mb, hipStream_t stream);
hipError_t wa_launch_row_write(const uint8_t* mask, int bh, int mb, int n, const int32_t* row_ptr, int32_t* col_idx,
                               hipStream_t stream);
