// Internal launch interface of the permutation kernels (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "wavealign.h"

struct WaPermLaunch {
  const uint64_t* rowbits;  // [bh][ceil(n/64)][m] word-major
  const uint64_t* colbits;  // [bh][ceil(m/64)][n] word-major
  const int32_t* row_nnz;   // [bh][m]
  int32_t* col_cnt;         // [bh][n], nullable
  int64_t* head_stats;      // [bh][6], nullable
  int32_t* perm;            // [bh][m]
  uint8_t* flags;           // [bh], nullable
  int32_t* embedding;       // [bh][m][2], nullable
  int32_t* stage1;          // [bh][m], nullable
  int32_t* seg_start;       // [bh][n_xcd+1], nullable
  int32_t bh, m, n;
  int32_t wave, n_xcd, iters, skip_mode, stats_only;
  int32_t block, head_dim;
  uint64_t seed;
  wa_skip_profile prof;
};

hipError_t wa_launch_perm_heads(const WaPermLaunch& a, hipStream_t stream);
size_t wa_perm_shared_bytes();
hipError_t wa_launch_fp64_probe(const double* a, const double* b, const int64_t* c, double* out, int n,
                                hipStream_t stream);
hipError_t wa_launch_pack_rows(const uint8_t* mask, int64_t rows, int m, int n, uint64_t* rowbits,
                               int32_t* row_nnz, hipStream_t stream);
hipError_t wa_launch_transpose_bits(const uint64_t* rowbits, int bh, int m, int n, uint64_t* colbits,
                                    hipStream_t stream);
hipError_t wa_launch_xcc_probe(int32_t* out, int n_wg, hipStream_t stream);
