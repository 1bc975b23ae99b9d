// Block-sparse attention forward for gfx950 (MI355X).
//
// One workgroup computes one query block (Sec. II-C: query blocks in the outer
// loop, the mask-selected KV blocks in the inner loop, the online-softmax state
// and partial O kept on chip). The workgroup has BLK/32 wavefronts; wavefront w
// owns query rows [32w, 32w+32) of the block.
//
// Per KV block j (ascending j, from the compacted list):
//   * the workgroup stages K_j row-major and V_j transposed (V^T[d][key]) in LDS;
//   * each wavefront computes S^T = K_j Q^T with v_mfma_f32_32x32x16_bf16
//     (A = K rows from LDS, B = its Q columns held in registers); in the MFMA
//     output layout a lane holds the scores of one query (lane mod 32) for 16
//     keys per 32-key tile, so the softmax max and sum are lane-local plus one
//     exchange with lane^32;
//   * the scores become P^T in bf16 in place: the accumulator registers of a
//     32-key tile, taken 8 at a time, are exactly the B operand of
//     O^T += V^T P^T when the contraction index runs over the keys in the order
//     the output layout holds them. The A operand (V^T rows) uses the same key
//     order, read as two 8-byte LDS loads from the transposed V tile;
//   * O^T is rescaled by exp2(m_old - m_new) before accumulation.
// At the end O = O^T / l is written at the block's original rows, which fuses
// the inverse permutation into the store.
//
// Workgroup -> query block: workgroup g of head bh runs slot xcd_slot(g) and
// slot s computes original block perm[s] (identity when perm is null).

#include "common.h"

namespace {

using wa::bf16x8;
using wa::f32x16;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __builtin_bit_cast(uint32_t, f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return (uint32_t)f32_to_bf16_rne(a) | ((uint32_t)f32_to_bf16_rne(b) << 16);
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

template <int D, int BLK>
__global__ __launch_bounds__(BLK * 2) void attn_fwd_kernel(WaAttnLaunch a) {
  constexpr int NW = BLK / 32;       // wavefronts per workgroup
  constexpr int NT = NW * 64;        // threads
  constexpr int KSTR = D + 8;        // K tile row stride (bf16 elements), 16-byte multiple
  constexpr int VSTR = BLK + 4;      // V^T tile row stride (bf16 elements), 8-byte multiple
  constexpr int KT = BLK / 32;       // 32-key tiles per KV block
  constexpr int DT = D / 32;         // 32-column tiles of O
  constexpr int KS = D / 16;         // k-steps of the QK^T product

  __shared__ __attribute__((aligned(16))) uint16_t ks_lds[BLK * KSTR];
  __shared__ __attribute__((aligned(16))) uint16_t vt_lds[D * VSTR];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int l32 = lane & 31;
  const int hf = lane >> 5;

  const int wgh = wa::wg_per_head(a.mb, a.n_xcd);
  const int bh = blockIdx.x / wgh;
  const int slot = wa::xcd_slot(blockIdx.x % wgh, a.mb, a.n_xcd);
  if (slot < 0) return;
  const int row = a.perm ? a.perm[(int64_t)bh * a.mb + slot] : slot;
  if ((unsigned)row >= (unsigned)a.mb) return;  // not a valid block index: nothing to compute

  const int n = a.seq_len;
  const uint16_t* qg = (const uint16_t*)a.q + (int64_t)bh * n * D;
  const uint16_t* kg = (const uint16_t*)a.k + (int64_t)bh * n * D;
  const uint16_t* vg = (const uint16_t*)a.v + (int64_t)bh * n * D;

  // Q columns for this wavefront: B operand of S^T = K Q^T.
  const int qi = row * BLK + w * 32 + l32;
  bf16x8 qf[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    uint4 val = make_uint4(0, 0, 0, 0);
    if (qi < n) val = *(const uint4*)(qg + (int64_t)qi * D + 16 * s + 8 * hf);
    qf[s] = as_bf16x8(val);
  }

  f32x16 oacc[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t)
#pragma unroll
    for (int v = 0; v < 16; ++v) oacc[t][v] = 0.f;

  float m_run = -INFINITY;
  float l_run = 0.f;
  const float c2 = a.scale * kLog2e;

  const int32_t* rp = a.row_ptr + (int64_t)bh * (a.mb + 1);
  const int beg = rp[row];
  const int end = rp[row + 1];
  const int32_t* cols = a.col_idx + (int64_t)bh * a.mb * a.mb;

  for (int e = beg; e < end; ++e) {
    const int j = cols[e];
    if ((unsigned)j >= (unsigned)a.mb) continue;  // uniform across the workgroup
    const int key0 = j * BLK;
    const int nvalid = min(BLK, n - key0);

    // ---- stage K_j (row-major) ----
    for (int c = tid; c < BLK * (D / 8); c += NT) {
      const int r = c / (D / 8), cc = c % (D / 8);
      uint4 val = make_uint4(0, 0, 0, 0);
      if (r < nvalid) val = *(const uint4*)(kg + (int64_t)(key0 + r) * D + cc * 8);
      *(uint4*)(ks_lds + r * KSTR + cc * 8) = val;
    }
    // ---- stage V_j transposed: task = (4 keys, 8 columns) ----
    for (int t = tid; t < (BLK / 4) * (D / 8); t += NT) {
      const int kq = t / (D / 8), dg = t % (D / 8);
      uint32_t wv[4][4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        uint4 val = make_uint4(0, 0, 0, 0);
        const int key = kq * 4 + r;
        if (key < nvalid) val = *(const uint4*)(vg + (int64_t)(key0 + key) * D + dg * 8);
        wv[r][0] = val.x; wv[r][1] = val.y; wv[r][2] = val.z; wv[r][3] = val.w;
      }
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const int sh = (c & 1) * 16;
        uint64_t e0 = (wv[0][c >> 1] >> sh) & 0xFFFFu;
        uint64_t e1 = (wv[1][c >> 1] >> sh) & 0xFFFFu;
        uint64_t e2 = (wv[2][c >> 1] >> sh) & 0xFFFFu;
        uint64_t e3 = (wv[3][c >> 1] >> sh) & 0xFFFFu;
        *(uint64_t*)(vt_lds + (dg * 8 + c) * VSTR + kq * 4) = e0 | (e1 << 16) | (e2 << 32) | (e3 << 48);
      }
    }
    __syncthreads();

    // ---- S^T = K_j Q^T ----
    f32x16 sacc[KT];
#pragma unroll
    for (int kt = 0; kt < KT; ++kt) {
#pragma unroll
      for (int v = 0; v < 16; ++v) sacc[kt][v] = 0.f;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const bf16x8 av = as_bf16x8(*(const uint4*)(ks_lds + (kt * 32 + l32) * KSTR + 16 * s + 8 * hf));
        sacc[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, qf[s], sacc[kt], 0, 0, 0);
      }
    }

    // ---- online softmax (log2 domain) ----
    if (nvalid < BLK) {
#pragma unroll
      for (int kt = 0; kt < KT; ++kt)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int key = kt * 32 + 8 * (v >> 2) + 4 * hf + (v & 3);
          if (key >= nvalid) sacc[kt][v] = -INFINITY;
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < KT; ++kt)
#pragma unroll
      for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sacc[kt][v]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx * c2);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    m_run = m_new;

    float lsum = 0.f;
    uint32_t pb[KT][8];
#pragma unroll
    for (int kt = 0; kt < KT; ++kt)
#pragma unroll
      for (int v = 0; v < 16; v += 2) {
        const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[kt][v], c2, -m_new));
        const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[kt][v + 1], c2, -m_new));
        lsum += p0 + p1;
        pb[kt][v >> 1] = pack_bf16x2(p0, p1);
      }
    l_run = l_run * alpha + lsum;
#pragma unroll
    for (int t = 0; t < DT; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) oacc[t][v] *= alpha;

    // ---- O^T += V^T P^T ----
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const uint16_t* vrow = vt_lds + (dt * 32 + l32) * VSTR + 4 * hf;
#pragma unroll
      for (int kt = 0; kt < KT; ++kt)
#pragma unroll
        for (int k2 = 0; k2 < 2; ++k2) {
          const int kb = kt * 32 + 16 * k2;
          uint2 lo = *(const uint2*)(vrow + kb);
          uint2 hi = *(const uint2*)(vrow + kb + 8);
          const bf16x8 av = as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y));
          const uint32_t* p = &pb[kt][4 * k2];
          const bf16x8 bv = as_bf16x8(make_uint4(p[0], p[1], p[2], p[3]));
          oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, oacc[dt], 0, 0, 0);
        }
    }
    __syncthreads();
  }

  // ---- epilogue: normalise and store at the original rows ----
  const float ltot = l_run + __shfl_xor(l_run, 32);
  const float inv = ltot > 0.f ? 1.f / ltot : 0.f;
  if (qi < n) {
    uint16_t* og = (uint16_t*)a.o + ((int64_t)bh * n + qi) * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int col = dt * 32 + 8 * g4 + 4 * hf;
        uint2 st;
        st.x = pack_bf16x2(oacc[dt][4 * g4 + 0] * inv, oacc[dt][4 * g4 + 1] * inv);
        st.y = pack_bf16x2(oacc[dt][4 * g4 + 2] * inv, oacc[dt][4 * g4 + 3] * inv);
        *(uint2*)(og + col) = st;
      }
    if (a.lse && hf == 0)
      a.lse[(int64_t)bh * n + qi] = ltot > 0.f ? (m_run + __log2f(ltot)) * kLn2 : -INFINITY;
  }
}

template <int D, int BLK>
hipError_t launch_t(const WaAttnLaunch& a, hipStream_t stream) {
  const int64_t grid = (int64_t)a.bh * wa::wg_per_head(a.mb, a.n_xcd);
  if (grid <= 0) return hipSuccess;
  hipLaunchKernelGGL((attn_fwd_kernel<D, BLK>), dim3((unsigned)grid), dim3(BLK * 2), 0, stream, a);
  return hipGetLastError();
}

template <int D, int BLK>
hipError_t occ_t(int* n) {
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(n, attn_fwd_kernel<D, BLK>, BLK * 2, 0);
}

}  // namespace

hipError_t wa_launch_attention(const WaAttnLaunch& a, hipStream_t stream) {
  if (a.head_dim == 128 && a.block == 128) return launch_t<128, 128>(a, stream);
  if (a.head_dim == 64 && a.block == 128) return launch_t<64, 128>(a, stream);
  if (a.head_dim == 128 && a.block == 64) return launch_t<128, 64>(a, stream);
  if (a.head_dim == 64 && a.block == 64) return launch_t<64, 64>(a, stream);
  return hipErrorInvalidValue;
}

hipError_t wa_attention_occupancy(int head_dim, int block, int* wgs_per_cu) {
  if (head_dim == 128 && block == 128) return occ_t<128, 128>(wgs_per_cu);
  if (head_dim == 64 && block == 128) return occ_t<64, 128>(wgs_per_cu);
  if (head_dim == 128 && block == 64) return occ_t<128, 64>(wgs_per_cu);
  if (head_dim == 64 && block == 64) return occ_t<64, 64>(wgs_per_cu);
  return hipErrorInvalidValue;
}
