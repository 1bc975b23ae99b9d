// Internal helpers shared by the HIP sources of the library (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// XCD segment [s0, s1) of a head: the entries x, x+1 of its segment table (clamped into [0, m] and
// made non-decreasing), or without a table n_xcd segments of equal row count, the first m mod n_xcd
// one row longer.
__host__ __device__ inline void xcd_segment(int x, int m, int n_xcd, const int32_t* seg, int* s0, int* s1) {
  if (seg) {
    const int a = min(max(seg[x], 0), m);
    *s0 = a;
    *s1 = min(max(seg[x + 1], a), m);
  } else {
    const int base = m / n_xcd, extra = m % n_xcd;
    *s0 = x * base + (x < extra ? x : extra);
    *s1 = *s0 + base + (x < extra ? 1 : 0);
  }
}

// Scheduler state of one attention call, in the caller's workspace: a task counter per queue
// (queue x holds segment x of every head, heads in order) and, per queue, the prefix sums of its
// segment lengths over the heads.
__host__ __device__ inline size_t sched_ints(int64_t bh, int n_xcd) { return 64 + (size_t)n_xcd * (bh + 1); }

// The last tail_heads(bh, m) heads of every queue run in an order built at each call (the tail
// order table, n_xcd x tail_heads x m int32 after the prefix tables): at most kTailEntries entries
// and kTailMaxHeads heads per queue.
constexpr int kTailEntries = 16384;
constexpr int kTailMaxHeads = 256;
__host__ __device__ inline int tail_heads(int64_t bh, int m) {
  if (bh <= 0 || m <= 0) return 0;
  int64_t w = kTailEntries / m;
  if (w > kTailMaxHeads) w = kTailMaxHeads;
  return (int)(bh < w ? bh : w);
}
__host__ __device__ inline size_t tail_offset(int64_t bh, int n_xcd) { return (sched_ints(bh, n_xcd) + 63) / 64 * 64; }
// Head-interleaved queue order (the alternative to heads in order): after the tail table, 64 queue
// offsets, then one entry h * m + slot per task, each queue's tasks round-robin over the heads.
__host__ __device__ inline size_t ilv_offset(int64_t bh, int m, int n_xcd) {
  return (tail_offset(bh, n_xcd) + (size_t)n_xcd * tail_heads(bh, m) * (m > 0 ? m : 0) + 63) / 64 * 64;
}
__host__ __device__ inline size_t sched_state_ints(int64_t bh, int m, int n_xcd) {
  return ilv_offset(bh, m, n_xcd) + 64 + (size_t)(bh > 0 ? bh : 0) * (m > 0 ? m : 0);
}

}  // namespace wa

// Launch helpers (implemented in the .hip sources, called by the ABI layer).
struct WaAttnLaunch {
  const void* q;
  const void* k;
  const void* v;     // null when the caller passes V already transposed (vt)
  void* vt;          // V transposed to [bh][head_dim][mb*block], zero-padded: the caller's, or the
                     // workspace copy that the launch writes from v
  int32_t* sched;    // workspace: sched_state_ints(bh, mb, n_xcd) int32 (counters at [0, n_xcd), prefix
                     // tables at 64, the tail order table at tail_offset(bh, n_xcd))
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
  int32_t head_order;  // 0 heads in order within each queue, 1 round-robin over the heads
  int32_t* status;     // device word, nullable: bit 0 an invalid perm entry, bit 1 an invalid KV index
  float scale;         // softmax scale
};

hipError_t wa_launch_attention(const WaAttnLaunch& a, hipStream_t stream);
// device address and size of the calling device's static scheduler scratch (looked up on first use)
hipError_t wa_noalloc_scratch(int32_t** ptr, size_t* bytes);
hipError_t wa_launch_transpose_v(const void* v, void* vt, int64_t bh, int seq_len, int mb, int head_dim, int block,
                                 hipStream_t stream);
hipError_t wa_attention_occupancy(int head_dim, int block, int* wgs_per_cu);
size_t wa_vt_bytes(int64_t bh, int mb, int head_dim, int block);

hipError_t wa_launch_row_count(const uint8_t* mask, int64_t rows, int n, int32_t* counts, int64_t count_stride_rows,
                               int counts_offset, int mb, hipStream_t stream);
hipError_t wa_launch_head_scan(int32_t* row_ptr, int bh, int mb, hipStream_t stream);
hipError_t wa_launch_row_write(const uint8_t* mask, int bh, int mb, int n, const int32_t* row_ptr, int32_t* col_idx,
                               hipStream_t stream);
