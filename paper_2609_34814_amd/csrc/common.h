// Internal helpers shared by the HIP sources of the library (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// Slot of workgroup `g` of one head under the XCD-aware mapping: workgroups are
// dispatched round-robin over the XCDs (g mod n_xcd), and XCD x runs the
// contiguous slot segment [seg_start(x), seg_start(x) + seg_len(x)) in order.
// Returns -1 for a workgroup with no slot (the last partial round).
__host__ __device__ inline int xcd_slot(int g, int m, int n_xcd) {
  if (n_xcd <= 1) return g < m ? g : -1;
  int x = g % n_xcd;
  int l = g / n_xcd;
  int base = m / n_xcd, extra = m % n_xcd;
  int len = base + (x < extra ? 1 : 0);
  if (l >= len) return -1;
  return x * base + (x < extra ? x : extra) + l;
}

__host__ __device__ inline int wg_per_head(int m, int n_xcd) {
  if (n_xcd <= 1) return m;
  return n_xcd * ((m + n_xcd - 1) / n_xcd);
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
