// Block-sparse attention forward for gfx950 (MI355X).
//
// One workgroup computes one query block (Sec. II-C: query blocks in the outer
// loop, the mask-selected KV blocks in the inner loop, the online-softmax state
// and partial O kept on chip). The workgroup has BLK/32 wavefronts; wavefront w
// owns query rows [32w, 32w+32) of the block. Two workgroups share a CU.
//
// Data movement. K_j and V_j^T (V transposed once per call into a zero-padded
// [d][N_pad] copy) are copied from global memory straight into LDS with
// global_load_lds_dwordx4 (no register staging; rows past the end of the
// sequence are clamped to the last row and masked). Only explicit vmcnt waits
// order these copies against LDS reads, so the copy into one tile stays in
// flight while the other tile is read. The LDS tiles are XOR-swizzled
// at 16-byte granularity so that the MFMA operand reads (ds_read_b128, one row
// per lane) are free of bank conflicts; the swizzle is applied by choosing each
// lane's global source chunk. The loads of K_{j+1} are issued as soon as every
// wavefront has finished reading K_j and overlap the softmax and P V of block j;
// the loads of V_{j+1} overlap the next Q K^T.
//
// Arithmetic (per wavefront, per KV block):
//   * S^T = K_j Q^T with v_mfma_f32_32x32x16_bf16: A = 32 key rows of K_j from
//     LDS, B = the wavefront's 32 query columns held in registers. MFMA row r of
//     a 32-key tile holds key 16(r/16) + pi(r mod 16), pi(4a+t) = {0,8,4,12}[a] + t,
//     so that in the output layout each lane holds, per 16 keys, 8 consecutive
//     keys of one query (lane mod 32): the softmax max and sum are lane-local plus
//     one exchange with lane^32, and
//   * P^T in bf16 is the B operand of O^T += V^T P^T directly from those
//     registers; the matching A operand is one 16-byte row chunk of V^T.
//   * O^T rows use the same permutation, so each lane finally holds 8 consecutive
//     output columns and O is written with 16-byte stores at the block's original
//     rows (the inverse permutation is fused into the store).
// Keys past the end of the sequence (ragged last block) get score -inf.
//
// Workgroup -> query blocks: workgroup g of head bh runs the slots xcd_slots(g)
// (its share of its XCD's segment) and slot s computes original block perm[s]
// (identity when perm is null).

#include "common.h"

#include <type_traits>

namespace {

using wa::bf16x8;
using wa::f32x16;

typedef __attribute__((address_space(3))) void lds_void_t;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kRescale = 8.0f;  // log2 headroom of the lazily rescaled running maximum

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding)
#define WA_WAIT_VM(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | (7 << 4) | (15 << 8) | (((n) >> 4) << 14))
// workgroup barrier after this wavefront's LDS reads have completed; the compiler may not move
// memory accesses across it
#define WA_BARRIER() asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory")

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// two floats -> two bf16 (round to nearest even; one v_cvt_pk_bf16_f32 on gfx950)
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  const f32x2 v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

// Row r (0..15) of an MFMA 16-row group -> tile row, so that the output layout
// gives each lane half 8 consecutive tile rows.
__device__ __forceinline__ int perm16(int r) { return ((r >> 2) & 1) * 8 + ((r >> 3) & 1) * 4 + (r & 3); }

// Tile with rows of RB bytes (256 or 128) in 16-byte chunks; physical chunk of (row, chunk).
template <int RB>
__device__ __forceinline__ int swz(int row, int chunk) {
  return RB == 256 ? (chunk ^ (row & 15)) : (chunk ^ ((row >> 1) & 7));
}

template <int RB>
__device__ __forceinline__ uint4 lds_chunk(const unsigned char* tile, int row, int chunk) {
  return *(const uint4*)(tile + row * RB + swz<RB>(row, chunk) * 16);
}

template <int D, int BLK>
struct Cfg {
  static constexpr int NW = BLK / 32;
  static constexpr int NT = NW * 64;
  static constexpr int KRB = D * 2;       // K tile row bytes
  static constexpr int VRB = BLK * 2;     // V^T tile row bytes
  static constexpr int KBYTES = BLK * KRB;
  static constexpr int VBYTES = D * VRB;
  static constexpr int NK = KBYTES / (NT * 16);  // DMA instructions per thread, K tile
  static constexpr int NV = VBYTES / (NT * 16);  // DMA instructions per thread, V^T tile
  static constexpr int KT = BLK / 32;
  static constexpr int DT = D / 32;
  static constexpr int KS = D / 16;
};

// One 16-byte-per-lane copy from global memory (uniform base + per-lane byte offset) into LDS at the
// uniform address lds (lane i writes lds + 16 i). Written as inline assembly so that only the
// explicit vmcnt waits of the pipeline order it against LDS reads of the other tile; M0 (the LDS
// base of the copy) is restored afterwards.
__device__ __forceinline__ void dma16(const void* gbase, uint32_t voff, const unsigned char* lds) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_void_t*)lds);
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "global_load_lds_dwordx4 %2, %3\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(m0), "v"(voff), "s"(gbase)
      : "memory");
}

// DMA geometry of a tile with rows of RB bytes copied by NW wavefronts: instruction i of wavefront w
// writes tile rows [(i*NW + w)*RPI, +RPI), lane l the chunk (l mod LPR) of row (l / LPR) among them.
// The global source of that slot is chunk swz(row, slot) of the row (the swizzle is an involution).
template <int RB, int NW>
struct Dma {
  static constexpr int RPI = 1024 / RB;   // rows per instruction
  static constexpr int LPR = RB / 16;     // lanes per row
  // the swizzle of a lane's slot is the same for every instruction when the row step is a multiple of 16
  static constexpr bool kInvariant = (NW * RPI) % 16 == 0;
  __device__ static __forceinline__ int row(int i, int w, int lane) { return (i * NW + w) * RPI + lane / LPR; }
  // per-lane source bytes relative to row (i*NW)*RPI of the tile (row stride `stride` bytes in memory)
  __device__ static __forceinline__ uint32_t lane_bytes(int i, int w, int lane, uint32_t stride) {
    const int r0 = w * RPI + lane / LPR;
    const int rs = kInvariant ? r0 : row(i, w, lane);
    return (uint32_t)r0 * stride + (uint32_t)(swz<RB>(rs, lane % LPR) * 16);
  }
};

// DMA of K rows [key0, key0 + BLK) of the head (kg: its first row) into the swizzled K tile. In the
// ragged last block, rows past the end of the sequence are clamped to the last row (their scores are
// masked).
template <int D, int BLK>
__device__ __forceinline__ void issue_k(unsigned char* ktile, const unsigned char* kg, int key0, int n, int w,
                                        int lane) {
  using C = Cfg<D, BLK>;
  using G = Dma<C::KRB, C::NW>;
  if (key0 + BLK <= n) {
#pragma unroll
    for (int i = 0; i < C::NK; ++i)
      dma16(kg + (int64_t)(key0 + i * C::NW * G::RPI) * C::KRB, G::lane_bytes(i, w, lane, C::KRB),
            ktile + (i * C::NW + w) * 1024);
  } else {
#pragma unroll
    for (int i = 0; i < C::NK; ++i) {
      const int r = G::row(i, w, lane);
      const uint32_t off = (uint32_t)min(key0 + r, n - 1) * (uint32_t)C::KRB +
                           (uint32_t)(swz<C::KRB>(r, lane % G::LPR) * 16);
      dma16(kg, off, ktile + (i * C::NW + w) * 1024);
    }
  }
}

// DMA of the V^T tile: rows d of the transposed copy (row stride row_bytes), keys [key0, key0 + BLK).
template <int D, int BLK>
__device__ __forceinline__ void issue_v(unsigned char* vtile, const unsigned char* vtg, uint32_t row_bytes, int key0,
                                        int w, int lane) {
  using C = Cfg<D, BLK>;
  using G = Dma<C::VRB, C::NW>;
#pragma unroll
  for (int i = 0; i < C::NV; ++i)
    dma16(vtg + (int64_t)key0 * 2 + (int64_t)(i * C::NW * G::RPI) * row_bytes, G::lane_bytes(i, w, lane, row_bytes),
          vtile + (i * C::NW + w) * 1024);
}

template <int D, int BLK>
__global__ __launch_bounds__(BLK * 2, 2) void attn_fwd_kernel(WaAttnLaunch a) {
  using C = Cfg<D, BLK>;
  __shared__ __attribute__((aligned(1024))) unsigned char k_lds[C::KBYTES];
  __shared__ __attribute__((aligned(1024))) unsigned char v_lds[C::VBYTES];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform within the wavefront
  const int l32 = lane & 31;
  const int hf = lane >> 5;

  const int wgh = wa::wg_per_head(a.mb, a.n_xcd);
  const int bh = blockIdx.x / wgh;
  int slot_first, slot_last;
  wa::xcd_slots(blockIdx.x % wgh, a.mb, a.n_xcd, a.seg ? a.seg + (int64_t)bh * (a.n_xcd + 1) : nullptr,
                &slot_first, &slot_last);
  for (int slot = slot_first; slot < slot_last; ++slot) {
  const int row = a.perm ? a.perm[(int64_t)bh * a.mb + slot] : slot;
  if ((unsigned)row >= (unsigned)a.mb) continue;  // not a valid block index: nothing to compute

  const int n = a.seq_len;
  const int64_t npad = (int64_t)a.mb * BLK;
  const uint16_t* qg = (const uint16_t*)a.q + (int64_t)bh * n * D;
  const unsigned char* kg = (const unsigned char*)a.k + (int64_t)bh * n * D * 2;
  const unsigned char* vtg = (const unsigned char*)a.vt + (int64_t)bh * D * npad * 2;
  const uint32_t vt_row_bytes = (uint32_t)(npad * 2);

  const int32_t* rp = a.row_ptr + (int64_t)bh * (a.mb + 1);
  const int beg = rp[row];
  const int end = rp[row + 1];
  // read-only for the whole kernel: the constant address space lets the list be read with scalar loads
  typedef const __attribute__((address_space(4))) int32_t* const_i32_ptr;
  const const_i32_ptr cols = (const_i32_ptr)(a.col_idx + (int64_t)bh * a.mb * a.mb);

  // Q columns of this wavefront: B operand of S^T = K Q^T
  const int qi = row * BLK + w * 32 + l32;
  bf16x8 qf[C::KS];
#pragma unroll
  for (int s = 0; s < C::KS; ++s) {
    uint4 val = make_uint4(0, 0, 0, 0);
    if (qi < n) val = *(const uint4*)(qg + (int64_t)qi * D + 16 * s + 8 * hf);
    qf[s] = as_bf16x8(val);
  }

  int j_cur = 0;
  if (beg < end) {
    j_cur = cols[beg];
    if ((unsigned)j_cur >= (unsigned)a.mb) j_cur = 0;
    issue_k<D, BLK>(k_lds, kg, j_cur * BLK, n, w, lane);
    issue_v<D, BLK>(v_lds, vtg, vt_row_bytes, j_cur * BLK, w, lane);
  }
  // the Q loads (issued first) are complete; the first tiles stay in flight
  WA_WAIT_VM(C::NK + C::NV);


  f32x16 oacc[C::DT];
#pragma unroll
  for (int t = 0; t < C::DT; ++t)
#pragma unroll
    for (int v = 0; v < 16; ++v) oacc[t][v] = 0.f;

  float m_run = -INFINITY;
  float l_run = 0.f;
  const float c2 = a.scale * kLog2e;
  const int krow_lane = 16 * (l32 >> 4) + perm16(l32 & 15);  // tile row supplied by this lane in a 32-row group

  // One KV block: wait for its tiles, S^T = K_j Q^T, online softmax, O^T += V_j^T P^T, and keep the
  // copies of the next block in flight. MASKED handles the ragged last block (keys past the end of
  // the sequence score -inf); the lists are ascending, so it can only be a row's last block.
  int e = beg;
  auto kv_block = [&](auto masked_tag) {
    constexpr bool MASKED = decltype(masked_tag)::value;
    const bool has_next = e + 1 < end;
    int j_next = 0;
    if (has_next) {
      j_next = cols[e + 1];
      if ((unsigned)j_next >= (unsigned)a.mb) j_next = 0;
    }

    // K_j resident (V_j may still be in flight)
    WA_WAIT_VM(C::NV);
    WA_BARRIER();

    // ---- S^T = K_j Q^T ----
    f32x16 sacc[C::KT];
#pragma unroll
    for (int kt = 0; kt < C::KT; ++kt) {
#pragma unroll
      for (int v = 0; v < 16; ++v) sacc[kt][v] = 0.f;
      const int krow = kt * 32 + krow_lane;
#pragma unroll
      for (int s = 0; s < C::KS; ++s) {
        const bf16x8 av = as_bf16x8(lds_chunk<C::KRB>(k_lds, krow, 2 * s + hf));
        sacc[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, qf[s], sacc[kt], 0, 0, 0);
      }
    }
    // every wavefront is done with K_j: start K_{j+1}
    WA_BARRIER();
    if (has_next) issue_k<D, BLK>(k_lds, kg, j_next * BLK, n, w, lane);

    // ---- online softmax (log2 domain) ----
    if constexpr (MASKED) {
      const int nvalid = n - j_cur * BLK;
#pragma unroll
      for (int kt = 0; kt < C::KT; ++kt)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int key = kt * 32 + 16 * (v >> 3) + 8 * hf + (v & 7);
          if (key >= nvalid) sacc[kt][v] = -INFINITY;
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < C::KT; ++kt)
#pragma unroll
      for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sacc[kt][v]);
    mx = fmaxf(mx, __shfl_xor(mx, 32)) * c2;
    // Lazy rescaling: the running maximum is raised (and O, l rescaled) only when some query of the
    // wavefront sees a score above it by more than kRescale; otherwise the probabilities are taken
    // against the old maximum and stay below 2^kRescale.
    if (__builtin_amdgcn_ballot_w64(mx > m_run + kRescale)) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int t = 0; t < C::DT; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) oacc[t][v] *= alpha;
    }

    float lsum = 0.f;
    uint32_t pb[C::KT][8];
#pragma unroll
    for (int kt = 0; kt < C::KT; ++kt)
#pragma unroll
      for (int v = 0; v < 16; v += 2) {
        const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[kt][v], c2, -m_run));
        const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[kt][v + 1], c2, -m_run));
        lsum += p0 + p1;
        pb[kt][v >> 1] = pack_bf16x2(p0, p1);
      }
    l_run += lsum;

    // V_j resident (K_{j+1} may still be in flight)
    if (has_next) {
      WA_WAIT_VM(C::NK);
    } else {
      WA_WAIT_VM(0);
    }
    WA_BARRIER();

    // ---- O^T += V_j^T P^T ----
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt) {
      const int vrow = dt * 32 + krow_lane;
#pragma unroll
      for (int kt = 0; kt < C::KT; ++kt)
#pragma unroll
        for (int k2 = 0; k2 < 2; ++k2) {
          const bf16x8 av = as_bf16x8(lds_chunk<C::VRB>(v_lds, vrow, 4 * kt + 2 * k2 + hf));
          const uint32_t* p = &pb[kt][4 * k2];
          const bf16x8 bv = as_bf16x8(make_uint4(p[0], p[1], p[2], p[3]));
          oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, oacc[dt], 0, 0, 0);
        }
    }
    // every wavefront is done with V_j: start V_{j+1}
    WA_BARRIER();
    if (has_next) issue_v<D, BLK>(v_lds, vtg, vt_row_bytes, j_next * BLK, w, lane);
    j_cur = j_next;
  };
  const bool ragged_last = end > beg && (n % BLK) != 0 && cols[end - 1] == a.mb - 1;
  for (; e < end - (ragged_last ? 1 : 0); ++e) kv_block(std::false_type{});
  if (ragged_last) kv_block(std::true_type{});

  // ---- epilogue: normalise and store at the original rows ----
  const float ltot = l_run + __shfl_xor(l_run, 32);
  const float inv = ltot > 0.f ? 1.f / ltot : 0.f;
  if (qi < n) {
    uint16_t* og = (uint16_t*)a.o + ((int64_t)bh * n + qi) * D;
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        const int col = dt * 32 + 16 * h2 + 8 * hf;
        uint4 st;
        st.x = pack_bf16x2(oacc[dt][8 * h2 + 0] * inv, oacc[dt][8 * h2 + 1] * inv);
        st.y = pack_bf16x2(oacc[dt][8 * h2 + 2] * inv, oacc[dt][8 * h2 + 3] * inv);
        st.z = pack_bf16x2(oacc[dt][8 * h2 + 4] * inv, oacc[dt][8 * h2 + 5] * inv);
        st.w = pack_bf16x2(oacc[dt][8 * h2 + 6] * inv, oacc[dt][8 * h2 + 7] * inv);
        *(uint4*)(og + col) = st;
      }
    if (a.lse && hf == 0)
      a.lse[(int64_t)bh * n + qi] = ltot > 0.f ? (m_run + __log2f(ltot)) * kLn2 : -INFINITY;
  }
  }  // slots
}

// V [bh][n][D] -> V^T [bh][D][mb*BLK], zero beyond n. One 64x64 tile per workgroup.
template <int D>
__global__ __launch_bounds__(256) void transpose_v_kernel(const uint16_t* __restrict__ v, uint16_t* __restrict__ vt,
                                                         int n, int64_t npad, int tiles_n) {
  __shared__ uint16_t t[64][66];
  const int tile = blockIdx.x % tiles_n;
  const int dtile = (blockIdx.x / tiles_n) % (D / 64);
  const int64_t bh = blockIdx.x / ((int64_t)tiles_n * (D / 64));
  const int key0 = tile * 64, d0 = dtile * 64;
  const uint16_t* src = v + bh * n * D;
  uint16_t* dst = vt + bh * D * npad;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int r = ty; r < 64; r += 4) {
    const int key = key0 + r;
    t[r][tx] = key < n ? src[(int64_t)key * D + d0 + tx] : (uint16_t)0;
  }
  __syncthreads();
  for (int r = ty; r < 64; r += 4) {
    const int64_t col = key0 + tx;
    if (col < npad) dst[(int64_t)(d0 + r) * npad + col] = t[tx][r];
  }
}

template <int D, int BLK>
hipError_t launch_t(const WaAttnLaunch& a, hipStream_t stream) {
  const int64_t npad = (int64_t)a.mb * BLK;
  const int tiles_n = (int)((npad + 63) / 64);
  const int64_t tgrid = (int64_t)a.bh * (D / 64) * tiles_n;
  hipLaunchKernelGGL((transpose_v_kernel<D>), dim3((unsigned)tgrid), dim3(256), 0, stream, (const uint16_t*)a.v,
                     (uint16_t*)a.vt, a.seq_len, npad, tiles_n);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
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

size_t wa_vt_bytes(int64_t bh, int mb, int head_dim, int block) {
  return (size_t)bh * head_dim * (size_t)mb * block * 2;
}

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
