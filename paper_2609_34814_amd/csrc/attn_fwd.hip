// Block-sparse attention forward for gfx950 (MI355X).
//
// One workgroup computes one query block (Sec. II-C: query blocks in the outer
// loop, the mask-selected KV blocks in the inner loop, the online-softmax state
// and partial O kept on chip). The workgroup has BLK/32 wavefronts; wavefront w
// owns query rows [32w, 32w+32) of the block. Two workgroups share a CU.
//
// Data movement. K_j (natural [token][d] layout) and V_j^T (from a transposed,
// zero-padded [d][N_pad] copy of V made once per call) are copied from global
// memory straight into LDS with global_load_lds_dwordx4 (no register staging;
// K rows past the end of the sequence are clamped to the last row and masked). Only explicit vmcnt waits order these copies against LDS
// reads, so the copy into one tile stays in flight while the other tile is read.
// The LDS tiles are XOR-swizzled at 16-byte granularity so that the MFMA operand
// reads are free of bank conflicts; the swizzle is applied by choosing each
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
//     registers; the matching A operand is one 16-byte row chunk of V^T (8 keys
//     of one d), so every operand read is one ds_read_b128. (Reading V in its
//     natural layout with ds_read_b64_tr_b16 takes two LDS instructions per
//     operand instead of one and measured slower.)
//   * O^T rows use the same permutation, so each lane finally holds 8 consecutive
//     output columns and O is written with 16-byte stores at the block's original
//     rows (the inverse permutation is fused into the store).
// Keys past the end of the sequence (ragged last block) get score -inf.
//
// Scheduling. The kernel is persistent: one workgroup per resident slot of the
// chip. Queue x holds, head after head, the slots of XCD segment x; a workgroup
// takes the next slot of the queue of the XCD it runs on (hardware XCC id), so
// that the query blocks that run together on one XCD, and share its L2, are
// consecutive slots of one segment (Sec. IV-D), and when that queue is empty
// it takes slots from the other queues. Slot s of head bh computes original
// query block perm[bh][s] (identity when perm is null). Row lengths are
// heavy-tailed (a row can hold ten times the mean number of blocks), and a launch
// whose last task is a long row ends with every other workgroup idle; so the last
// heads of each queue run in an order built at each call: a row that could still
// be running once the rest of the queue is done starts first, longest first, and
// every other row keeps its place (tail_order_kernel).

#include "common.h"
#include "wavealign.h"

#include <algorithm>
#include <mutex>
#include <type_traits>

namespace {

using wa::bf16x8;
using wa::f32x16;

typedef __attribute__((address_space(3))) void lds_void_t;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
// Probabilities are taken against the first block's row maximum; a row in which one reaches this
// bound is recomputed against its exact maximum (fp32 and bf16 hold values up to it exactly scaled).
constexpr float kProbLimit = 4294967296.0f;  // 2^32

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding)
#define WA_WAIT_VM(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | (7 << 4) | (15 << 8) | (((n) >> 4) << 14))
// workgroup barrier after this wavefront's LDS reads have completed; the compiler may not move
// memory accesses across it
#define WA_BARRIER() asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory")

// Scheduling fence: no instruction moves across it. Placed between the operand reads of k-step s+1
// and the MFMAs of k-step s, it keeps those reads in flight while the MFMAs run (left alone, the
// scheduler sinks every read to just before its MFMA, and each MFMA then waits out an LDS latency).
#define WA_SCHED_FENCE() __builtin_amdgcn_sched_barrier(0)

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

// Tiles have rows of RB bytes (256 or 128) in 16-byte chunks. Physical chunk of (row, chunk):
// K tiles are read one row per lane (ds_read_b128), 16 rows per wavefront quarter;
// V tiles are read by the transposing loads, four consecutive rows at a time.
template <int RB>
__device__ __forceinline__ int swz_k(int row, int chunk) {
  return RB == 256 ? (chunk ^ (row & 15)) : (chunk ^ ((row >> 1) & 7));
}
template <int RB>
__device__ __forceinline__ int swz_v(int row, int chunk) {
  const int e = row & 3;  // XOR 0, 6, 12, 10 (256-byte rows) or 0, 2, 4, 6 (128-byte rows): stays in the row
  return RB == 256 ? (chunk ^ ((e << 1) ^ (e << 2))) : (chunk ^ (e << 1));
}
template <int RB, bool V>
__device__ __forceinline__ int swz(int row, int chunk) {
  return V ? swz_v<RB>(row, chunk) : swz_k<RB>(row, chunk);
}

template <int RB>
__device__ __forceinline__ uint4 lds_chunk(const unsigned char* tile, int row, int chunk) {
  return *(const uint4*)(tile + row * RB + swz_k<RB>(row, chunk) * 16);
}

template <int D, int BLK>
struct Cfg {
  static constexpr int NW = BLK / 32;
  static constexpr int NT = NW * 64;
  static constexpr int RB = D * 2;        // K tile row bytes
  static constexpr int VRB = BLK * 2;     // V^T tile row bytes (one row per d)
  static constexpr int TBYTES = BLK * RB;  // K tile bytes = V^T tile bytes
  static constexpr int NK = TBYTES / (NT * 16);  // DMA instructions per thread and tile
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
// The global source of that slot is chunk swz(row, slot) of the row (each swizzle is an involution).
template <int RB, int NW, bool V>
struct Dma {
  static constexpr int RPI = 1024 / RB;   // rows per instruction
  static constexpr int LPR = RB / 16;     // lanes per row
  // the swizzle of a lane's slot is the same for every instruction when the row step is a multiple of
  // the swizzle's row period
  static constexpr bool kInvariant = (NW * RPI) % (V ? 4 : 16) == 0;
  __device__ static __forceinline__ int row(int i, int w, int lane) { return (i * NW + w) * RPI + lane / LPR; }
  // per-lane source bytes relative to tile row (i*NW)*RPI, for source rows `stride` bytes apart
  __device__ static __forceinline__ uint32_t lane_bytes(int i, int w, int lane, uint32_t stride = RB) {
    const int r0 = w * RPI + lane / LPR;
    const int rs = kInvariant ? r0 : row(i, w, lane);
    return (uint32_t)r0 * stride + (uint32_t)(swz<RB, V>(rs, lane % LPR) * 16);
  }
};

// DMA of rows [key0, key0 + BLK) of a K or V head (g: its first row) into a swizzled tile. In the
// ragged last block, rows past the end of the sequence are clamped to the last row (their scores
// are masked, so their probabilities are 0).
template <int D, int BLK, bool V>
__device__ __forceinline__ void issue_tile(unsigned char* tile, const unsigned char* g, int key0, int n, int w,
                                           int lane) {
  using C = Cfg<D, BLK>;
  using G = Dma<C::RB, C::NW, V>;
  if (key0 + BLK <= n) {
#pragma unroll
    for (int i = 0; i < C::NK; ++i)
      dma16(g + (int64_t)(key0 + i * C::NW * G::RPI) * C::RB, G::lane_bytes(i, w, lane),
            tile + (i * C::NW + w) * 1024);
  } else {
#pragma unroll
    for (int i = 0; i < C::NK; ++i) {
      const int r = G::row(i, w, lane);
      const uint32_t off = (uint32_t)min(key0 + r, n - 1) * (uint32_t)C::RB +
                           (uint32_t)(swz<C::RB, V>(r, lane % G::LPR) * 16);
      dma16(g, off, tile + (i * C::NW + w) * 1024);
    }
  }
}

// DMA of the V^T tile: rows d of the transposed copy (row stride row_bytes), keys [key0, key0 + BLK),
// into a tile with the K-tile swizzle (rows of VRB bytes, read one row chunk per lane).
template <int D, int BLK>
__device__ __forceinline__ void issue_vt(unsigned char* tile, const unsigned char* vtg, uint32_t row_bytes, int key0,
                                         int w, int lane) {
  using C = Cfg<D, BLK>;
  using G = Dma<C::VRB, C::NW, false>;
#pragma unroll
  for (int i = 0; i < C::NK; ++i)
    dma16(vtg + (int64_t)key0 * 2 + (int64_t)(i * C::NW * G::RPI) * row_bytes, G::lane_bytes(i, w, lane, row_bytes),
          tile + (i * C::NW + w) * 1024);
}

// Next task of this workgroup: slot of a head from the queue of its XCD, else from the others.
// Run by one lane; returns false when every queue is exhausted.
__device__ bool fetch_task(const WaAttnLaunch& a, int home, int* bh_out, int* slot_out) {
  int32_t* cnt = a.sched;
  const int32_t* pre = a.sched + 64;
  const int th = wa::tail_heads(a.bh, a.mb);
  for (int k = 0; k < a.n_xcd; ++k) {
    const int x = (home + k) % a.n_xcd;
    const int32_t* px = pre + (int64_t)x * (a.bh + 1);
    const int total = px[a.bh];
    if (__hip_atomic_load(cnt + x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= total) continue;
    const int t = atomicAdd(cnt + x, 1);
    if (t >= total) continue;
    if (a.head_order) {  // round-robin over the heads: the call's order table
      const int32_t* ilv = a.sched + wa::ilv_offset(a.bh, a.mb, a.n_xcd);
      const int ent = ilv[64 + ilv[x] + t];
      *bh_out = ent / a.mb;
      *slot_out = ent - *bh_out * a.mb;
      return true;
    }
    const int tb = px[a.bh - th];
    if (t >= tb) {  // the last heads: the call's tail order
      const int e = a.sched[wa::tail_offset(a.bh, a.n_xcd) + (int64_t)x * th * a.mb + (t - tb)];
      *bh_out = a.bh - th + (e >> 16);
      *slot_out = e & 0xFFFF;
      return true;
    }
    // head h with px[h] <= t < px[h+1]
    int lo = 0, hi = a.bh - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (px[mid] <= t) lo = mid; else hi = mid - 1;
    }
    int s0, s1;
    wa::xcd_segment(x, a.mb, a.n_xcd, a.seg ? a.seg + (int64_t)lo * (a.n_xcd + 1) : nullptr, &s0, &s1);
    *bh_out = lo;
    *slot_out = s0 + (t - px[lo]);
    return true;
  }
  return false;
}

template <int D, int BLK>
__global__ __launch_bounds__(BLK * 2, 2) void attn_fwd_kernel(WaAttnLaunch a) {
  using C = Cfg<D, BLK>;
  __shared__ __attribute__((aligned(1024))) unsigned char k_lds[C::TBYTES];
  __shared__ __attribute__((aligned(1024))) unsigned char v_lds[C::TBYTES];
  __shared__ int task[2];
  __shared__ int redo;  // the current row is recomputed against its exact maximum

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform within the wavefront
  const int l32 = lane & 31;
  const int hf = lane >> 5;
  const int n = a.seq_len;
  const float c2 = a.scale * kLog2e;

  const int home = (int)(__builtin_amdgcn_s_getreg((3 << 11) | (0 << 6) | 20) & 0xF) % a.n_xcd;
  // byte offsets of this lane's K-operand chunk of k-step s in the K tile (key tile kt adds kt 32 RB)
  uint32_t kofs[C::KS];
  {
    const int kr = 16 * ((lane & 31) >> 4) + perm16(lane & 15);
#pragma unroll
    for (int s = 0; s < C::KS; ++s) kofs[s] = (uint32_t)(kr * C::RB + swz_k<C::RB>(kr, 2 * s + hf) * 16);
  }
  // the same for the V^T operand of k-step ks (16 keys; d tile dt adds dt 32 VRB)
  uint32_t vofs[2 * C::KT];
  {
    const int kr = 16 * ((lane & 31) >> 4) + perm16(lane & 15);
#pragma unroll
    for (int ks = 0; ks < 2 * C::KT; ++ks)
      vofs[ks] = (uint32_t)(kr * C::VRB + swz_k<C::VRB>(kr, 2 * ks + hf) * 16);
  }

  for (;;) {
    if (tid == 0) {
      int tb = -1, ts = 0;
      if (!fetch_task(a, home, &tb, &ts)) tb = -1;
      task[0] = tb;
      task[1] = ts;
      redo = 0;
    }
    __syncthreads();
    const int bh = __builtin_amdgcn_readfirstlane(task[0]);
    const int slot = __builtin_amdgcn_readfirstlane(task[1]);
    __syncthreads();  // every wavefront has read the task before it is overwritten
    if (bh < 0) break;
    const int row = a.perm ? a.perm[(int64_t)bh * a.mb + slot] : slot;
    if ((unsigned)row >= (unsigned)a.mb) {  // not a valid block index: nothing to compute, reported
      if (tid == 0 && a.status) atomicOr(a.status, 1);
      continue;
    }

    const uint16_t* qg = (const uint16_t*)a.q + (int64_t)bh * n * D;
    const unsigned char* kg = (const unsigned char*)a.k + (int64_t)bh * n * D * 2;
    const int64_t npad = (int64_t)a.mb * BLK;
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

    f32x16 oacc[C::DT];
    int bad_kv = 0;           // the row's list held an index outside 0..mb-1 (uniform)
    float m_run = -INFINITY;  // reference maximum (log2 units), set by the row's first block
    float l_run = 0.f;
    int j_cur = 0;

    // S^T = K_j Q^T from the K tile in LDS. Consecutive MFMAs go to different accumulators (a chain on
    // one accumulator would wait for each result), and the operand reads of k-step s+1 are in flight
    // during the MFMAs of step s.
    auto scores = [&](f32x16 (&sacc)[C::KT]) {
#pragma unroll
      for (int kt = 0; kt < C::KT; ++kt)
#pragma unroll
        for (int v = 0; v < 16; ++v) sacc[kt][v] = 0.f;
      uint4 a_cur[C::KT], a_nxt[C::KT];
#pragma unroll
      for (int kt = 0; kt < C::KT; ++kt) a_cur[kt] = *(const uint4*)(k_lds + kofs[0] + kt * 32 * C::RB);
#pragma unroll
      for (int s = 0; s < C::KS; ++s) {
        if (s + 1 < C::KS) {
#pragma unroll
          for (int kt = 0; kt < C::KT; ++kt) a_nxt[kt] = *(const uint4*)(k_lds + kofs[s + 1] + kt * 32 * C::RB);
        }
        WA_SCHED_FENCE();
#pragma unroll
        for (int kt = 0; kt < C::KT; ++kt)
          sacc[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a_cur[kt]), qf[s], sacc[kt], 0, 0, 0);
        WA_SCHED_FENCE();
#pragma unroll
        for (int kt = 0; kt < C::KT; ++kt) a_cur[kt] = a_nxt[kt];
      }
    };
    // keys past the end of the sequence (ragged last block) score -inf
    auto mask_tail = [&](f32x16 (&sacc)[C::KT], int nvalid, int lane_o) {
      const int hf_o = lane_o >> 5;  // from the opaque lane copy: no key table held across blocks
#pragma unroll
      for (int kt = 0; kt < C::KT; ++kt)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int key = kt * 32 + 16 * (v >> 3) + 8 * hf_o + (v & 7);
          if (key >= nvalid) sacc[kt][v] = -INFINITY;
        }
    };
    // row maximum of a score tile, in log2 units (shared by the two lanes of a query)
    auto tile_max = [&](const f32x16 (&sacc)[C::KT]) {
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < C::KT; ++kt)
#pragma unroll
        for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sacc[kt][v]);
      return fmaxf(mx, __shfl_xor(mx, 32)) * c2;
    };

    // One KV block: wait for its tiles, S^T = K_j Q^T, softmax numerators, O^T += V_j^T P^T, and keep
    // the copies of the next block in flight. MASKED handles the ragged last block; the lists are
    // ascending, so it can only be a row's last block. FIRST takes the block's row maximum as the
    // softmax reference of the row: every later probability is taken against it, so O and l are never
    // rescaled (a row whose probabilities outgrow the reference is recomputed, below).
    int e = beg;
    auto kv_block = [&](auto masked_tag, auto first_tag) {
      constexpr bool MASKED = decltype(masked_tag)::value;
      constexpr bool FIRST = decltype(first_tag)::value;
      // The per-lane copy offsets are recomputed in every block from an opaque copy of the lane index
      // (hoisted out of the loop they would hold registers that the operand reads need); the operand
      // read offsets, one per k-step, are computed once per kernel (kofs, vofs).
      int lane_o = lane;
      asm volatile("" : "+v"(lane_o));
      const bool has_next = e + 1 < end;
      int j_next = 0;
      if (has_next) {
        j_next = cols[e + 1];
        if ((unsigned)j_next >= (unsigned)a.mb) {  // invalid KV index: block 0 is read, reported
          j_next = 0;
          bad_kv = 1;
        }
      }

      // K_j resident (V_j may still be in flight)
      WA_WAIT_VM(C::NK);
      WA_BARRIER();
      f32x16 sacc[C::KT];
      scores(sacc);
      // every wavefront is done with K_j: start K_{j+1}
      WA_BARRIER();
      if (has_next) issue_tile<D, BLK, false>(k_lds, kg, j_next * BLK, n, w, lane_o);

      // ---- softmax numerators (log2 domain) ----
      if constexpr (MASKED) mask_tail(sacc, n - j_cur * BLK, lane_o);
      if constexpr (FIRST) m_run = tile_max(sacc);
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
      {
        // k-step ks = 2 kt + k2 (16 keys); operand reads of step ks+1 in flight during step ks
        uint4 a_cur[C::DT], a_nxt[C::DT];
#pragma unroll
        for (int dt = 0; dt < C::DT; ++dt) a_cur[dt] = *(const uint4*)(v_lds + vofs[0] + dt * 32 * C::VRB);
#pragma unroll
        for (int ks = 0; ks < 2 * C::KT; ++ks) {
          if (ks + 1 < 2 * C::KT) {
#pragma unroll
            for (int dt = 0; dt < C::DT; ++dt)
              a_nxt[dt] = *(const uint4*)(v_lds + vofs[ks + 1] + dt * 32 * C::VRB);
          }
          const uint32_t* p = &pb[ks >> 1][4 * (ks & 1)];
          const bf16x8 bv = as_bf16x8(make_uint4(p[0], p[1], p[2], p[3]));
#pragma unroll
          for (int dt = 0; dt < C::DT; ++dt)
            oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a_cur[dt]), bv, oacc[dt], 0, 0, 0);
#pragma unroll
          for (int dt = 0; dt < C::DT; ++dt) a_cur[dt] = a_nxt[dt];
        }
      }
      // every wavefront is done with V_j: start V_{j+1}
      WA_BARRIER();
      if (has_next) issue_vt<D, BLK>(v_lds, vtg, vt_row_bytes, j_next * BLK, w, lane_o);
      j_cur = j_next;
    };
    const bool ragged_last = end > beg && (n % BLK) != 0 && cols[end - 1] == a.mb - 1;
    const int e_plain = end - (ragged_last ? 1 : 0);

    // Pass 0 takes the first block's maximum as the reference. If some probability reached
    // kProbLimit (a later score above the reference by log2(kProbLimit) or more, in log2 units), the
    // whole workgroup recomputes the row: the exact row maximum over all its blocks first, then
    // pass 1 against it (every probability <= 1). The decision is per workgroup, since its wavefronts
    // share the tile copies.
    for (int pass = 0;; ++pass) {
      if (beg < end) {
        j_cur = cols[beg];
        if ((unsigned)j_cur >= (unsigned)a.mb) {
          j_cur = 0;
          bad_kv = 1;
        }
        issue_tile<D, BLK, false>(k_lds, kg, j_cur * BLK, n, w, lane);
        issue_vt<D, BLK>(v_lds, vtg, vt_row_bytes, j_cur * BLK, w, lane);
      }
      // the Q loads (issued first) are complete; the first tiles stay in flight
      WA_WAIT_VM(2 * C::NK);
#pragma unroll
      for (int t = 0; t < C::DT; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) oacc[t][v] = 0.f;
      l_run = 0.f;
      e = beg;
      if (e < e_plain) {
        if (pass == 0) {
          kv_block(std::false_type{}, std::true_type{});
        } else {
          kv_block(std::false_type{}, std::false_type{});
        }
        for (++e; e < e_plain; ++e) kv_block(std::false_type{}, std::false_type{});
        if (ragged_last) kv_block(std::true_type{}, std::false_type{});
      } else if (ragged_last) {
        if (pass == 0) {
          kv_block(std::true_type{}, std::true_type{});
        } else {
          kv_block(std::true_type{}, std::false_type{});
        }
      }
      if (pass > 0) break;
      if (__builtin_amdgcn_ballot_w64(!(l_run < kProbLimit)) && lane == 0) redo = 1;  // also inf / NaN
      __syncthreads();
      const int again = __builtin_amdgcn_readfirstlane(redo);
      __syncthreads();  // every wavefront has read the flag before the next row clears it
      if (!again) break;
      // exact row maximum: K tiles one at a time, scores only
      float mx = -INFINITY;
      for (int e2 = beg; e2 < end; ++e2) {
        int j = cols[e2];
        if ((unsigned)j >= (unsigned)a.mb) j = 0;
        issue_tile<D, BLK, false>(k_lds, kg, j * BLK, n, w, lane);
        WA_WAIT_VM(0);
        WA_BARRIER();
        f32x16 sacc[C::KT];
        scores(sacc);
        if (j * BLK + BLK > n) mask_tail(sacc, n - j * BLK, lane);
        mx = fmaxf(mx, tile_max(sacc));
        WA_BARRIER();  // every wavefront is done with the tile before the next copy
      }
      m_run = mx;
    }

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
    if (bad_kv && tid == 0 && a.status) atomicOr(a.status, 2);
  }
}

// Scheduler set-up: zero the queue counters and the status word, and build, per queue, the prefix
// sums of its segment lengths over the heads. One workgroup; thread x handles queue x.
__global__ __launch_bounds__(64) void sched_kernel(int32_t* sched, const int32_t* seg, int32_t* status, int bh,
                                                   int mb, int n_xcd) {
  const int x = threadIdx.x;
  if (x == 0 && status) *status = 0;
  if (x >= n_xcd) return;
  sched[x] = 0;
  int32_t* px = sched + 64 + (int64_t)x * (bh + 1);
  int acc = 0;
  px[0] = 0;
  for (int h = 0; h < bh; ++h) {
    int s0, s1;
    wa::xcd_segment(x, mb, n_xcd, seg ? seg + (int64_t)h * (n_xcd + 1) : nullptr, &s0, &s1);
    acc += s1 - s0;
    px[h + 1] = acc;
  }
}

// Tail order of queue x (one workgroup per queue): entries e = 0, 1, ... enumerate, in queue order,
// the slots of segment x of the last th heads. A row of n blocks that starts with fewer than
// 2 n (grid / n_xcd) blocks queued after it could outlast the rest of the queue; such rows go first,
// by descending n (ties in queue order), and the others follow in queue order. Each entry is
// (head offset << 16) | slot. The order is a permutation of the queue's slots, so every row still
// runs exactly once.
__global__ __launch_bounds__(1024) void tail_order_kernel(WaAttnLaunch a, int grid) {
  constexpr int NT = 1024;
  constexpr int PER = wa::kTailEntries / NT;
  __shared__ int32_t hstart[wa::kTailMaxHeads + 1];  // first entry of each head's segment
  __shared__ int32_t hslot0[wa::kTailMaxHeads];      // its first slot
  __shared__ int32_t part[NT];
  __shared__ uint32_t key[wa::kTailEntries];
  const int x = blockIdx.x;
  const int t = threadIdx.x;
  const int th = wa::tail_heads(a.bh, a.mb);
  const int hb = a.bh - th;
  int32_t* tail = a.sched + wa::tail_offset(a.bh, a.n_xcd) + (int64_t)x * th * a.mb;
  if (t < th) {
    int s0, s1;
    wa::xcd_segment(x, a.mb, a.n_xcd, a.seg ? a.seg + (int64_t)(hb + t) * (a.n_xcd + 1) : nullptr, &s0, &s1);
    hslot0[t] = s0;
    part[t] = s1 - s0;
  }
  __syncthreads();
  if (t == 0) {
    int acc = 0;
    for (int k = 0; k < th; ++k) {
      hstart[k] = acc;
      acc += part[k];
    }
    hstart[th] = acc;
  }
  __syncthreads();
  const int total = hstart[th];
  // head offset of entry e: the last k with hstart[k] <= e
  auto head_of = [&](int e) {
    int lo = 0, hi = th - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (hstart[mid] <= e) lo = mid; else hi = mid - 1;
    }
    return lo;
  };
  // block counts of this thread's entries PER t .. PER t + PER - 1 (independent loads first)
  int row[PER], nb[PER];
  const int e0 = t * PER;
  int k = e0 < total ? head_of(e0) : 0;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int e = e0 + i;
    row[i] = -1;
    if (e < total) {
      while (e >= hstart[k + 1]) ++k;
      const int slot = hslot0[k] + (e - hstart[k]);
      row[i] = a.perm ? a.perm[(int64_t)(hb + k) * a.mb + slot] : slot;
    }
  }
  k = e0 < total ? head_of(e0) : 0;
  int sum = 0;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int e = e0 + i;
    nb[i] = 0;
    if (e < total) {
      while (e >= hstart[k + 1]) ++k;
      if ((unsigned)row[i] < (unsigned)a.mb) {
        const int32_t* rp = a.row_ptr + (int64_t)(hb + k) * (a.mb + 1);
        nb[i] = min(max(rp[row[i] + 1] - rp[row[i]], 0), WA_MAX_BLOCKS);
      }
    }
    sum += nb[i];
  }
  // blocks queued after each entry, then the late entries and their ranks (block-wide scans)
  auto block_scan = [&](int v, int* all) {  // inclusive prefix sum over the threads, and the total
    part[t] = v;
    __syncthreads();
    for (int off = 1; off < NT; off <<= 1) {
      const int u = t >= off ? part[t - off] : 0;
      __syncthreads();
      part[t] += u;
      __syncthreads();
    }
    const int r = part[t];
    *all = part[NT - 1];
    __syncthreads();
    return r;
  };
  const int64_t wgs = max(grid / a.n_xcd, 1);
  int all = 0;
  const int incl = block_scan(sum, &all);
  int64_t after = (int64_t)all - incl;  // blocks of the entries after this thread's
  uint32_t late_bits = 0;
  int nlate_mine = 0;
#pragma unroll
  for (int i = PER - 1; i >= 0; --i) {
    const int e = e0 + i;
    if (e < total && 2 * (int64_t)nb[i] * wgs > after) {
      late_bits |= 1u << i;
      ++nlate_mine;
    }
    after += nb[i];
  }
  int nlate = 0;
  const int late_incl = block_scan(nlate_mine, &nlate);
  int late_before = late_incl - nlate_mine;
  int P = 1;
  while (P < nlate) P <<= 1;
  for (int i = t; i < P; i += NT) key[i] = 0xFFFFFFFFu;
  __syncthreads();
  k = e0 < total ? head_of(e0) : 0;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int e = e0 + i;
    if (e < total) {
      while (e >= hstart[k + 1]) ++k;
      if (late_bits >> i & 1u) {
        key[late_before++] = ((uint32_t)(WA_MAX_BLOCKS - nb[i]) << 14) | (uint32_t)e;
      } else {
        tail[nlate + (e - late_before)] = (k << 16) | (hslot0[k] + (e - hstart[k]));
      }
    }
  }
  __syncthreads();
  // late entries: bitonic sort ascending = descending block count, ties in queue order
  for (int kk = 2; kk <= P; kk <<= 1)
    for (int j = kk >> 1; j > 0; j >>= 1) {
      for (int i = t; i < P; i += NT) {
        const int l = i ^ j;
        if (l > i) {
          const uint32_t u = key[i], v = key[l];
          if ((u > v) == ((i & kk) == 0)) {
            key[i] = v;
            key[l] = u;
          }
        }
      }
      __syncthreads();
    }
  for (int i = t; i < nlate; i += NT) {
    const int e = (int)(key[i] & 0x3FFFu);
    const int kh = head_of(e);
    tail[i] = (kh << 16) | (hslot0[kh] + (e - hstart[kh]));
  }
}

// Head-interleaved order of queue x (one workgroup per queue): the queue's tasks round-robin over the
// heads, round r taking slot s0_h + r of every head h whose segment of the queue has more than r
// slots, heads ascending. Entry (h, r) therefore sits at C(r) + #{h' < h : L_h' > r}, with L_h the
// segment length and C(r) = sum_h min(L_h, r) the entries of the rounds before r. Entries are
// h * mb + slot; queue x's entries start at the total of queues 0..x-1 (ilv[x]).
__global__ __launch_bounds__(1024) void ilv_order_kernel(WaAttnLaunch a) {
  constexpr int NT = 1024;
  constexpr int RPT = WA_MAX_BLOCKS / NT;  // rounds per thread: r = t + k NT < mb <= WA_MAX_BLOCKS
  __shared__ int off_s;
  const int x = blockIdx.x;
  const int t = threadIdx.x;
  int32_t* ilv = a.sched + wa::ilv_offset(a.bh, a.mb, a.n_xcd);
  if (t == 0) {
    int off = 0;
    for (int y = 0; y < x; ++y) off += a.sched[64 + (int64_t)y * (a.bh + 1) + a.bh];
    ilv[x] = off;
    off_s = off;
  }
  __syncthreads();
  int32_t* out = ilv + 64 + off_s;
  int c[RPT];
#pragma unroll
  for (int k = 0; k < RPT; ++k) c[k] = 0;
  for (int h = 0; h < a.bh; ++h) {
    int s0, s1;
    wa::xcd_segment(x, a.mb, a.n_xcd, a.seg ? a.seg + (int64_t)h * (a.n_xcd + 1) : nullptr, &s0, &s1);
#pragma unroll
    for (int k = 0; k < RPT; ++k) c[k] += min(s1 - s0, t + k * NT);
  }
  for (int h = 0; h < a.bh; ++h) {
    int s0, s1;
    wa::xcd_segment(x, a.mb, a.n_xcd, a.seg ? a.seg + (int64_t)h * (a.n_xcd + 1) : nullptr, &s0, &s1);
#pragma unroll
    for (int k = 0; k < RPT; ++k) {
      const int r = t + k * NT;
      if (r < s1 - s0) out[c[k]++] = h * a.mb + s0 + r;
    }
  }
}

// V [bh][n][D] -> V^T [bh][D][npad], zero for keys >= n. One 64-key x 64-column tile per workgroup,
// 16-byte loads and stores, transposed through LDS.
template <int D>
__global__ __launch_bounds__(256) void transpose_v_kernel(const uint16_t* __restrict__ v, uint16_t* __restrict__ vt,
                                                         int n, int64_t npad, int tiles_n) {
  __shared__ uint16_t t[64][64 + 8];
  const int tile = blockIdx.x % tiles_n;
  const int dtile = (blockIdx.x / tiles_n) % (D / 64);
  const int64_t bh = blockIdx.x / ((int64_t)tiles_n * (D / 64));
  const int key0 = tile * 64, d0 = dtile * 64;
  const uint16_t* src = v + bh * n * D;
  uint16_t* dst = vt + bh * D * npad;
  const int tid = threadIdx.x;
  // load: thread -> (key r, 8-column group c8), two passes of 32 keys
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    const int r = pass * 32 + tid / 8, c8 = tid % 8;
    uint4 val = make_uint4(0, 0, 0, 0);
    if (key0 + r < n) val = *(const uint4*)(src + (int64_t)(key0 + r) * D + d0 + c8 * 8);
    const uint32_t wv[4] = {val.x, val.y, val.z, val.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) t[r][c8 * 8 + e] = (uint16_t)(wv[e >> 1] >> ((e & 1) * 16));
  }
  __syncthreads();
  // store: thread -> (column d, 8-key group k8), two passes of 32 columns
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    const int d = pass * 32 + tid / 8, k8 = tid % 8;
    uint32_t wv[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      wv[e] = (uint32_t)t[k8 * 8 + 2 * e][d] | ((uint32_t)t[k8 * 8 + 2 * e + 1][d] << 16);
    *(uint4*)(dst + (int64_t)(d0 + d) * npad + key0 + k8 * 8) = make_uint4(wv[0], wv[1], wv[2], wv[3]);
  }
}

int resident_cus() {
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

template <int D>
hipError_t launch_transpose(const void* v, void* vt, int64_t bh, int n, int mb, int blk, hipStream_t stream) {
  const int64_t npad = (int64_t)mb * blk;
  const int tiles_n = (int)((npad + 63) / 64);
  const int64_t tgrid = bh * (D / 64) * tiles_n;
  if (tgrid <= 0) return hipSuccess;
  hipLaunchKernelGGL((transpose_v_kernel<D>), dim3((unsigned)tgrid), dim3(256), 0, stream, (const uint16_t*)v,
                     (uint16_t*)vt, n, npad, tiles_n);
  return hipGetLastError();
}

template <int D, int BLK>
hipError_t launch_t(const WaAttnLaunch& a, hipStream_t stream) {
  hipLaunchKernelGGL(sched_kernel, dim3(1), dim3(64), 0, stream, a.sched, a.seg, a.status, a.bh, a.mb, a.n_xcd);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t tasks = (int64_t)a.bh * a.mb;
  int occ = 0;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, attn_fwd_kernel<D, BLK>, BLK * 2, 0);
  if (e != hipSuccess) return e;
  const int64_t grid = std::min<int64_t>(tasks, (int64_t)resident_cus() * std::max(occ, 1));
  if (tasks > 0) {
    if (a.head_order) {
      hipLaunchKernelGGL(ilv_order_kernel, dim3(a.n_xcd), dim3(1024), 0, stream, a);
    } else {
      hipLaunchKernelGGL(tail_order_kernel, dim3(a.n_xcd), dim3(1024), 0, stream, a, (int)grid);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (a.v) {  // V given in its natural layout: the call's transposed copy
    e = launch_transpose<D>(a.v, a.vt, a.bh, a.seq_len, a.mb, BLK, stream);
    if (e != hipSuccess) return e;
  }
  if (tasks <= 0) return hipSuccess;
  hipLaunchKernelGGL((attn_fwd_kernel<D, BLK>), dim3((unsigned)grid), dim3(BLK * 2), 0, stream, a);
  return hipGetLastError();
}

template <int D, int BLK>
hipError_t occ_t(int* n) {
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(n, attn_fwd_kernel<D, BLK>, BLK * 2, 0);
}

}  // namespace

// Scheduler state of the attention entry point that allocates nothing: a static device array of the
// library, one per GPU, held until the process ends. Host code never uses the array's name as an
// address: its device address is looked up once per device (with that device current) and cached.
static constexpr size_t kNoAllocInts = WA_NOALLOC_SCRATCH_BYTES / 4;
static __device__ __align__(256) int32_t scratch[kNoAllocInts];
static std::mutex g_scratch_mu;
static int32_t* g_scratch_ptr[64];

hipError_t wa_noalloc_scratch(int32_t** ptr, size_t* bytes) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = (int32_t*)p;
  }
  *ptr = g_scratch_ptr[dev];
  *bytes = kNoAllocInts * 4;
  return hipSuccess;
}

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

hipError_t wa_launch_transpose_v(const void* v, void* vt, int64_t bh, int seq_len, int mb, int head_dim, int block,
                                 hipStream_t stream) {
  if (head_dim == 128) return launch_transpose<128>(v, vt, bh, seq_len, mb, block, stream);
  if (head_dim == 64) return launch_transpose<64>(v, vt, bh, seq_len, mb, block, stream);
  return hipErrorInvalidValue;
}

hipError_t wa_attention_occupancy(int head_dim, int block, int* wgs_per_cu) {
  if (head_dim == 128 && block == 128) return occ_t<128, 128>(wgs_per_cu);
  if (head_dim == 64 && block == 128) return occ_t<64, 128>(wgs_per_cu);
  if (head_dim == 128 && block == 64) return occ_t<128, 64>(wgs_per_cu);
  if (head_dim == 64 && block == 64) return occ_t<64, 64>(wgs_per_cu);
  return hipErrorInvalidValue;
}
