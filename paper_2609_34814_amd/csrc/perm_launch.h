// Internal launch interface of the permutation kernels (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "wavealign.h"

// Per-head state carried between the permutation kernels (workspace, 64 bytes a head).
struct PermState {
  uint64_t maxy;    // max |Ym| of the current centred product (atomic max over column slices)
  int32_t active;   // the subspace iteration still runs for this head
  int32_t degen;    // a QR found no direction
  int32_t done;     // the init kernel already wrote this head's result (skipped head)
  int32_t flags;    // skip-rule flags of cases 1-3
  int64_t nnz, sum_c2;
  int64_t adj_and, adj_or;  // adjacent-row overlap of the natural order: sum |M_i & M_i+1|, sum |M_i | M_i+1|
  int64_t pad[1];
};
static_assert(sizeof(PermState) == 64, "PermState is 64 bytes");

struct WaPermLaunch {
  const uint64_t* rowbits;  // [bh][ceil(n/64)][m] word-major
  const uint64_t* colbits;  // [bh][ceil(m/64)][n] word-major
  const int32_t* row_nnz;   // [bh][m]
  int32_t* cc;              // workspace [bh][n]: column counts
  int32_t* col_cnt;         // [bh][n], nullable (a copy of the column counts for the caller)
  int32_t* xg;              // workspace [bh][m][2]: X of the subspace iteration (2^30 fixed point)
  int64_t* ym;              // workspace [bh][n][2]: m * M~^T X
  int64_t* z;               // workspace [bh][m][2]: m * M~ Ys
  PermState* state;         // workspace [bh]
  int64_t* head_stats;      // [bh][6], nullable
  int32_t* perm;            // [bh][m]
  uint8_t* flags;           // [bh], nullable
  int32_t* embedding;       // [bh][m][2], nullable
  int32_t* stage1;          // [bh][m], nullable
  int32_t* seg_start;       // [bh][n_xcd+1], nullable
  int32_t bh, m, n, slices;
  int32_t wave, n_xcd, iters, skip_mode, stats_only;
  int32_t block, head_dim;
  uint64_t seed;
  wa_skip_profile prof;
};

hipError_t wa_launch_perm(const WaPermLaunch& a, hipStream_t stream);
size_t wa_perm_shared_bytes();
int wa_perm_slices(int n);  // workgroups per head of the centred-product kernels (n: the larger of m, n)
hipError_t wa_launch_fp64_probe(const double* a, const double* b, const int64_t* c, double* out, int n,
                                hipStream_t stream);
hipError_t wa_launch_pack_rows(const uint8_t* mask, int64_t rows, int m, int n, uint64_t* rowbits,
                               int32_t* row_nnz, hipStream_t stream);
hipError_t wa_launch_transpose_bits(const uint64_t* rowbits, int bh, int m, int n, uint64_t* colbits,
                                    hipStream_t stream);
hipError_t wa_launch_xcc_probe(int32_t* out, int n_wg, hipStream_t stream);
hipError_t wa_launch_check_perm(const int32_t* perm, int bh, int m, int32_t* bad, int32_t* head_ok,
                                hipStream_t stream);
