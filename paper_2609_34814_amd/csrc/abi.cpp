// C ABI of the library: argument validation, workspace layout and kernel dispatch.
// Every argument is checked before any HIP call; nothing here allocates or synchronises.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "common.h"
#include "perm_launch.h"
#include "producer_launch.h"
#include "wavealign.h"

namespace {

thread_local char g_err[512] = "";

wa_status fail(wa_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return s;
}

wa_status ok() {
  g_err[0] = '\0';
  return WA_OK;
}

wa_status hip_fail(hipError_t e, const char* what) {
  return fail(WA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

struct Dims {
  int64_t bh;
  int mb;
  int n;  // tokens
  int d;
  int blk;
};

wa_status check_shape(const wa_shape* s, Dims* out) {
  if (!s) return fail(WA_ERR_INVALID_ARG, "shape is null");
  if (s->batch < 1 || s->heads < 1 || s->seq_len < 1)
    return fail(WA_ERR_INVALID_ARG, "batch, heads and seq_len must be >= 1 (got %d, %d, %d)", s->batch, s->heads,
                s->seq_len);
  if (s->head_dim != 64 && s->head_dim != 128)
    return fail(WA_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", s->head_dim);
  if (s->block != 64 && s->block != 128)
    return fail(WA_ERR_UNSUPPORTED, "block %d not supported (64 or 128)", s->block);
  const int64_t mb = ((int64_t)s->seq_len + s->block - 1) / s->block;
  if (mb > WA_MAX_BLOCKS) return fail(WA_ERR_UNSUPPORTED, "%lld blocks per sequence exceeds %d", (long long)mb,
                                      WA_MAX_BLOCKS);
  const int64_t bh = (int64_t)s->batch * s->heads;
  if (bh * mb * mb >= (int64_t(1) << 31))
    return fail(WA_ERR_UNSUPPORTED, "batch*heads*M_B*N_B = %lld must be < 2^31", (long long)(bh * mb * mb));
  if (bh * (int64_t)s->seq_len * s->head_dim >= (int64_t(1) << 40))
    return fail(WA_ERR_UNSUPPORTED, "tensor too large");
  out->bh = bh;
  out->mb = (int)mb;
  out->n = s->seq_len;
  out->d = s->head_dim;
  out->blk = s->block;
  return WA_OK;
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

struct ProducerWs {
  size_t means, amax, bmax, codes, queue, total;
};

ProducerWs producer_ws_layout(const Dims& d) {
  ProducerWs w{};
  size_t off = 0;
  w.means = off; off = align_up(off + (size_t)2 * d.bh * d.mb * d.d * 4);
  w.amax = off; off = align_up(off + (size_t)2 * d.bh * 4);
  w.bmax = off; off = align_up(off + (size_t)2 * d.bh * d.mb * 4);
  w.codes = off; off = align_up(off + (size_t)2 * d.bh * d.mb * d.d);
  w.queue = off; off = align_up(off + (size_t)wa_producer_queue_words(d.bh) * 4);
  w.total = off;
  return w;
}

struct PermWs {
  size_t rowbits, colbits, row_nnz, col_cnt, head_stats, xg, ym, z, state, total;
  int slices;
};

PermWs perm_ws_layout(const Dims& d) {
  PermWs w{};
  const int64_t words = (d.mb + 63) / 64;
  w.slices = wa_perm_slices(d.mb);
  size_t off = 0;
  w.rowbits = off; off = align_up(off + (size_t)d.bh * d.mb * words * 8);
  w.colbits = off; off = align_up(off + (size_t)d.bh * d.mb * words * 8);
  w.row_nnz = off; off = align_up(off + (size_t)d.bh * d.mb * 4);
  w.col_cnt = off; off = align_up(off + (size_t)d.bh * d.mb * 4);
  w.head_stats = off; off = align_up(off + (size_t)d.bh * 6 * 8);
  w.xg = off; off = align_up(off + (size_t)d.bh * d.mb * 2 * 4);
  w.ym = off; off = align_up(off + (size_t)d.bh * d.mb * 2 * 8);
  w.z = off; off = align_up(off + (size_t)d.bh * d.mb * 2 * 8);
  w.state = off; off = align_up(off + (size_t)d.bh * sizeof(PermState));
  w.total = off;
  return w;
}

void perm_ws_pointers(WaPermLaunch& a, const PermWs& L, char* base) {
  a.rowbits = (const uint64_t*)(base + L.rowbits);
  a.colbits = (const uint64_t*)(base + L.colbits);
  a.cc = (int32_t*)(base + L.col_cnt);
  a.xg = (int32_t*)(base + L.xg);
  a.ym = (int64_t*)(base + L.ym);
  a.z = (int64_t*)(base + L.z);
  a.state = (PermState*)(base + L.state);
  a.slices = L.slices;
}

// Attention workspace: [scheduler state][V^T copy][row_ptr][col_idx]; the CSR entry point uses the
// first two parts. The scheduler part is sized for the largest n_xcd.
constexpr int kMaxXcd = 64;
size_t attn_sched_bytes(const Dims& d) { return align_up(wa::sched_state_ints(d.bh, d.mb, kMaxXcd) * 4); }
size_t attn_csr_ws_bytes(const Dims& d) {
  return attn_sched_bytes(d) + align_up(wa_vt_bytes(d.bh, d.mb, d.d, d.blk));
}
size_t attn_ws_bytes(const Dims& d) {
  return attn_csr_ws_bytes(d) + align_up((size_t)d.bh * (d.mb + 1) * 4) + align_up((size_t)d.bh * d.mb * d.mb * 4);
}

wa_status check_ws(void* ws, size_t have, size_t need) {
  if (need == 0) return WA_OK;
  if (!ws) return fail(WA_ERR_INVALID_ARG, "workspace is null (%zu bytes needed)", need);
  if (!aligned(ws, kAlign)) return fail(WA_ERR_ALIGNMENT, "workspace must be 256-byte aligned");
  if (have < need) return fail(WA_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", have, need);
  return WA_OK;
}

// MI355X offline profiles from the sequence-length and density sweep of the attention step.
const wa_skip_profile kDefaultProfile = {
    96.0 * 1024.0 * 1024.0,  // cache_bytes: K/V per head below which reordering did not pay (the shared
                             // 256 MiB last-level cache holds it next to the streamed Q, O and V^T)
    0.5,                     // gain_ns_per_block: attention time saved per kept block where it paid
    -3000.0,                 // ovh_ns_fixed    } permutation time per head of more than 1024 blocks (the
    11.06,                   // ovh_ns_per_row  } sliced form), amortised over concurrent heads, least-
    0.0,                     // ovh_ns_per_nnz  } squares fit over 1,547-4,079 blocks (worst residual 11%)
    0.2,                     // j_max: adjacent rows of raster-local heads share 23-40% of their blocks
    0.05,                    // eta_min
    1024.0,                  // fused_max_blocks: heads built by one workgroup (the matrix-core form)
    1184.0,                  // ovh_fused_ns_fixed   } the one-workgroup form's time per head, fitted alone
    10.50,                   // ovh_fused_ns_per_row } (worst residual 3%)
    0.0,                     // ovh_fused_ns_per_nnz }
};

wa_status check_attn_common(const void* q, const void* k, const void* v, void* o, int32_t n_xcd, float* lse,
                            int32_t* status) {
  if (!q || !k || !v || !o) return fail(WA_ERR_INVALID_ARG, "q, k, v and o must be non-null");
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(o, 16))
    return fail(WA_ERR_ALIGNMENT, "q, k, v and o must be 16-byte aligned");
  if (n_xcd < 1 || n_xcd > kMaxXcd) return fail(WA_ERR_INVALID_ARG, "n_xcd %d outside 1..%d", n_xcd, kMaxXcd);
  if (lse && !aligned(lse, 4)) return fail(WA_ERR_ALIGNMENT, "lse must be 4-byte aligned");
  if (status && !aligned(status, 4)) return fail(WA_ERR_ALIGNMENT, "status must be 4-byte aligned");
  return WA_OK;
}

wa_status launch_compact(const uint8_t* mask, const Dims& d, int32_t* row_ptr, int32_t* col_idx, hipStream_t st) {
  hipError_t e = wa_launch_row_count(mask, d.bh * d.mb, d.mb, row_ptr, d.mb + 1, 1, d.mb, st);
  if (e != hipSuccess) return hip_fail(e, "row_count launch");
  e = wa_launch_head_scan(row_ptr, (int)d.bh, d.mb, st);
  if (e != hipSuccess) return hip_fail(e, "head_scan launch");
  e = wa_launch_row_write(mask, (int)d.bh, d.mb, d.mb, row_ptr, col_idx, st);
  if (e != hipSuccess) return hip_fail(e, "row_write launch");
  return WA_OK;
}

// v: V in its natural layout (transposed into the workspace after the scheduler state), or null with
// vt: V already transposed by the caller.
wa_status launch_attn(const void* q, const void* k, const void* v, const void* vt, void* ws, const int32_t* row_ptr,
                      const int32_t* col_idx, const int32_t* perm, const int32_t* seg, const Dims& d, float scale,
                      int32_t n_xcd, int32_t head_order, void* o, float* lse, int32_t* status, hipStream_t st) {
  WaAttnLaunch a{};
  a.q = q; a.k = k; a.v = v;
  a.sched = (int32_t*)ws;
  a.vt = v ? (void*)((char*)ws + attn_sched_bytes(d)) : const_cast<void*>(vt);
  a.row_ptr = row_ptr; a.col_idx = col_idx; a.perm = perm; a.seg = seg;
  a.o = o; a.lse = lse; a.status = status; a.head_order = head_order;
  a.bh = (int32_t)d.bh; a.seq_len = d.n; a.mb = d.mb; a.head_dim = d.d; a.block = d.blk; a.n_xcd = n_xcd;
  a.scale = (scale > 0.f && std::isfinite(scale)) ? scale : (float)(1.0 / std::sqrt((double)d.d));
  hipError_t e = wa_launch_attention(a, st);
  if (e != hipSuccess) return hip_fail(e, "attention launch");
  return WA_OK;
}

wa_status perm_launch_common(const uint8_t* mask, const Dims& d, const PermWs& L, char* base, hipStream_t st,
                             int32_t* row_nnz_out) {
  int32_t* row_nnz = row_nnz_out ? row_nnz_out : (int32_t*)(base + L.row_nnz);
  hipError_t e = wa_launch_pack_rows(mask, d.bh * d.mb, d.mb, d.mb, (uint64_t*)(base + L.rowbits), row_nnz, st);
  if (e != hipSuccess) return hip_fail(e, "pack_rows launch");
  e = wa_launch_transpose_bits((const uint64_t*)(base + L.rowbits), (int)d.bh, d.mb, d.mb,
                               (uint64_t*)(base + L.colbits), st);
  if (e != hipSuccess) return hip_fail(e, "transpose_bits launch");
  return WA_OK;
}

}  // namespace

extern "C" {

int32_t wa_abi_version(void) { return WA_ABI_VERSION; }

const char* wa_status_string(wa_status s) {
  switch (s) {
    case WA_OK: return "ok";
    case WA_ERR_INVALID_ARG: return "invalid argument";
    case WA_ERR_UNSUPPORTED: return "unsupported shape or parameter";
    case WA_ERR_ALIGNMENT: return "misaligned pointer";
    case WA_ERR_WORKSPACE: return "workspace too small";
    case WA_ERR_INVALID_PERM: return "not a permutation";
    case WA_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char* wa_last_error(void) { return g_err; }

wa_status wa_default_skip_profile(wa_skip_profile* out) {
  if (!out) return fail(WA_ERR_INVALID_ARG, "out is null");
  *out = kDefaultProfile;
  return ok();
}

wa_status wa_wave_size(int32_t head_dim, int32_t block, int32_t* wave_per_xcd) {
  if (!wave_per_xcd) return fail(WA_ERR_INVALID_ARG, "wave_per_xcd is null");
  if ((head_dim != 64 && head_dim != 128) || (block != 64 && block != 128))
    return fail(WA_ERR_UNSUPPORTED, "head_dim %d / block %d not supported", head_dim, block);
  int dev = 0, cus = 0, wgs = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute");
  e = wa_attention_occupancy(head_dim, block, &wgs);
  if (e != hipSuccess) return hip_fail(e, "occupancy query");
  // 8 XCDs share the compute units evenly on MI355X (256 CUs = 8 x 32)
  const int per_xcd = cus >= 8 ? cus / 8 : cus;
  *wave_per_xcd = per_xcd * (wgs > 0 ? wgs : 1);
  return ok();
}

wa_status wa_perm_workspace_size(const wa_shape* shape, size_t* bytes) {
  Dims d;
  wa_status s = check_shape(shape, &d);
  if (s != WA_OK) return s;
  if (!bytes) return fail(WA_ERR_INVALID_ARG, "bytes is null");
  *bytes = perm_ws_layout(d).total;
  return ok();
}

wa_status wa_mask_stats(const uint8_t* mask, const wa_shape* shape, int32_t* row_nnz, int32_t* col_cnt,
                        int64_t* head_stats, void* workspace, size_t workspace_bytes, void* stream) {
  Dims d;
  wa_status s = check_shape(shape, &d);
  if (s != WA_OK) return s;
  if (!mask || !row_nnz || !col_cnt || !head_stats)
    return fail(WA_ERR_INVALID_ARG, "mask, row_nnz, col_cnt and head_stats must be non-null");
  const PermWs L = perm_ws_layout(d);
  s = check_ws(workspace, workspace_bytes, L.total);
  if (s != WA_OK) return s;
  hipStream_t st = (hipStream_t)stream;
  char* base = (char*)workspace;
  s = perm_launch_common(mask, d, L, base, st, row_nnz);
  if (s != WA_OK) return s;
  WaPermLaunch a{};
  perm_ws_pointers(a, L, base);
  a.row_nnz = row_nnz;
  a.col_cnt = col_cnt;
  a.head_stats = head_stats;
  a.bh = (int32_t)d.bh; a.m = d.mb; a.n = d.mb;
  a.wave = 1; a.n_xcd = 1; a.iters = 0; a.skip_mode = WA_SKIP_NEVER; a.stats_only = 1;
  a.block = d.blk; a.head_dim = d.d;
  a.prof = kDefaultProfile;
  hipError_t e = wa_launch_perm(a, st);
  if (e != hipSuccess) return hip_fail(e, "mask stats launch");
  return ok();
}

wa_status wa_build_permutation(const uint8_t* mask, const wa_shape* shape, const wa_perm_params* params,
                               int32_t* perm, int32_t* seg_start, uint8_t* head_flags, int32_t* embedding,
                               int32_t* stage1_order, void* workspace, size_t workspace_bytes, void* stream) {
  Dims d;
  wa_status s = check_shape(shape, &d);
  if (s != WA_OK) return s;
  if (!params) return fail(WA_ERR_INVALID_ARG, "params is null");
  if (!mask || !perm) return fail(WA_ERR_INVALID_ARG, "mask and perm must be non-null");
  if (params->n_xcd < 1 || params->n_xcd > 64) return fail(WA_ERR_INVALID_ARG, "n_xcd %d outside 1..64", params->n_xcd);
  if (params->iters < 1 || params->iters > 64) return fail(WA_ERR_INVALID_ARG, "iters %d outside 1..64", params->iters);
  if (params->skip_mode < WA_SKIP_AUTO || params->skip_mode > WA_SKIP_ALWAYS)
    return fail(WA_ERR_INVALID_ARG, "skip_mode %d invalid", params->skip_mode);
  if (params->wave_per_xcd < 0 || params->wave_per_xcd > WA_MAX_BLOCKS)
    return fail(WA_ERR_INVALID_ARG, "wave_per_xcd %d outside 0..%d", params->wave_per_xcd, WA_MAX_BLOCKS);
  if (embedding && !aligned(embedding, 8)) return fail(WA_ERR_ALIGNMENT, "embedding must be 8-byte aligned");
  const PermWs L = perm_ws_layout(d);
  s = check_ws(workspace, workspace_bytes, L.total);
  if (s != WA_OK) return s;
  int32_t wave = params->wave_per_xcd;
  if (wave == 0) {
    s = wa_wave_size(d.d, d.blk, &wave);
    if (s != WA_OK) return s;
  }
  hipStream_t st = (hipStream_t)stream;
  char* base = (char*)workspace;
  s = perm_launch_common(mask, d, L, base, st, nullptr);
  if (s != WA_OK) return s;
  WaPermLaunch a{};
  perm_ws_pointers(a, L, base);
  a.row_nnz = (const int32_t*)(base + L.row_nnz);
  a.col_cnt = nullptr;
  a.head_stats = nullptr;
  a.perm = perm; a.flags = head_flags; a.embedding = embedding; a.stage1 = stage1_order; a.seg_start = seg_start;
  a.bh = (int32_t)d.bh; a.m = d.mb; a.n = d.mb;
  a.wave = wave; a.n_xcd = params->n_xcd; a.iters = params->iters; a.skip_mode = params->skip_mode;
  a.stats_only = 0; a.block = d.blk; a.head_dim = d.d; a.seed = params->seed;
  a.prof = params->profile ? *params->profile : kDefaultProfile;
  hipError_t e = wa_launch_perm(a, st);
  if (e != hipSuccess) return hip_fail(e, "permutation launch");
  return ok();
}

wa_status wa_mask_producer_workspace_size(const wa_shape* shape, size_t* bytes) {
  Dims d;
  wa_status s = check_shape(shape, &d);
  if (s != WA_OK) return s;
  if (!bytes) return fail(WA_ERR_INVALID_ARG, "bytes is null");
  *bytes = producer_ws_layout(d).total;
  return ok();
}

wa_status wa_produce_block_mask(const void* q, const void* k, const wa_shape* shape, int32_t keep, int32_t diagonal,
                                uint8_t* mask, int8_t* codes, int32_t* status, void* workspace,
                                size_t workspace_bytes, void* stream) {
  Dims d;
  wa_status s = check_shape(shape, &d);
  if (s != WA_OK) return s;
  if (!q || !k || !mask) return fail(WA_ERR_INVALID_ARG, "q, k and mask must be non-null");
  if (keep < 0) return fail(WA_ERR_INVALID_ARG, "keep %d is negative", keep);
  if (!aligned(q, 16) || !aligned(k, 16)) return fail(WA_ERR_ALIGNMENT, "q and k must be 16-byte aligned");
  if (codes && !aligned(codes, 16)) return fail(WA_ERR_ALIGNMENT, "codes must be 16-byte aligned");
  if (status && !aligned(status, 4)) return fail(WA_ERR_ALIGNMENT, "status must be 4-byte aligned");
  const ProducerWs L = producer_ws_layout(d);
  s = check_ws(workspace, workspace_bytes, L.total);
  if (s != WA_OK) return s;
  char* base = (char*)workspace;
  WaProducerLaunch a{};
  a.q = q; a.k = k;
  a.means = (float*)(base + L.means);
  a.amax = (uint32_t*)(base + L.amax);
  a.bmax = (uint32_t*)(base + L.bmax);
  a.codes = codes ? codes : (int8_t*)(base + L.codes);
  a.mask = mask;
  a.queue = (uint32_t*)(base + L.queue);
  a.status = status;
  a.bh = (int32_t)d.bh; a.mb = d.mb; a.seq_len = d.n; a.block = d.blk; a.head_dim = d.d;
  a.keep = keep; a.diagonal = diagonal ? 1 : 0;
  hipError_t e = wa_launch_producer(a, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "mask producer launch");
  return ok();
}

wa_status wa_check_perm_workspace_size(const wa_shape* shape, size_t* bytes) {
  Dims d;
  wa_status s = check_shape(shape, &d);
  if (s != WA_OK) return s;
  if (!bytes) return fail(WA_ERR_INVALID_ARG, "bytes is null");
  *bytes = kAlign;
  return ok();
}

wa_status wa_check_perm(const int32_t* perm, const wa_shape* shape, int32_t* head_ok, void* workspace,
                        size_t workspace_bytes, void* stream) {
  Dims d;
  wa_status s = check_shape(shape, &d);
  if (s != WA_OK) return s;
  if (!perm) return fail(WA_ERR_INVALID_ARG, "perm is null");
  s = check_ws(workspace, workspace_bytes, kAlign);
  if (s != WA_OK) return s;
  hipStream_t st = (hipStream_t)stream;
  int32_t* bad = (int32_t*)workspace;
  hipError_t e = wa_launch_check_perm(perm, (int)d.bh, d.mb, bad, head_ok, st);
  if (e != hipSuccess) return hip_fail(e, "check_perm launch");
  int32_t host_bad = 0;
  e = hipMemcpyAsync(&host_bad, bad, sizeof(host_bad), hipMemcpyDeviceToHost, st);
  if (e != hipSuccess) return hip_fail(e, "check_perm copy");
  e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hip_fail(e, "check_perm synchronize");
  if (host_bad != 0)
    return fail(WA_ERR_INVALID_PERM, "%d of %lld heads hold no permutation of 0..%d", host_bad, (long long)d.bh,
                d.mb - 1);
  return ok();
}

wa_status wa_compact_mask(const uint8_t* mask, const wa_shape* shape, int32_t* row_ptr, int32_t* col_idx,
                          void* stream) {
  Dims d;
  wa_status s = check_shape(shape, &d);
  if (s != WA_OK) return s;
  if (!mask || !row_ptr || !col_idx) return fail(WA_ERR_INVALID_ARG, "mask, row_ptr and col_idx must be non-null");
  s = launch_compact(mask, d, row_ptr, col_idx, (hipStream_t)stream);
  if (s != WA_OK) return s;
  return ok();
}

wa_status wa_attn_workspace_size(const wa_shape* shape, size_t* bytes) {
  Dims d;
  wa_status s = check_shape(shape, &d);
  if (s != WA_OK) return s;
  if (!bytes) return fail(WA_ERR_INVALID_ARG, "bytes is null");
  *bytes = attn_ws_bytes(d);
  return ok();
}

wa_status wa_sparse_attn(const void* q, const void* k, const void* v, const uint8_t* mask, const int32_t* perm,
                         const int32_t* seg_start, const wa_shape* shape, float softmax_scale, int32_t n_xcd,
                         void* o, float* lse, int32_t* status, void* workspace, size_t workspace_bytes,
                         void* stream) {
  Dims d;
  wa_status s = check_shape(shape, &d);
  if (s != WA_OK) return s;
  s = check_attn_common(q, k, v, o, n_xcd, lse, status);
  if (s != WA_OK) return s;
  if (!mask) return fail(WA_ERR_INVALID_ARG, "mask is null");
  s = check_ws(workspace, workspace_bytes, attn_ws_bytes(d));
  if (s != WA_OK) return s;
  hipStream_t st = (hipStream_t)stream;
  char* base = (char*)workspace;
  int32_t* row_ptr = (int32_t*)(base + attn_csr_ws_bytes(d));
  int32_t* col_idx = (int32_t*)(base + attn_csr_ws_bytes(d) + align_up((size_t)d.bh * (d.mb + 1) * 4));
  s = launch_compact(mask, d, row_ptr, col_idx, st);
  if (s != WA_OK) return s;
  s = launch_attn(q, k, v, nullptr, base, row_ptr, col_idx, perm, seg_start, d, softmax_scale, n_xcd, 0, o, lse,
                  status, st);
  if (s != WA_OK) return s;
  return ok();
}

wa_status wa_sparse_attn_csr(const void* q, const void* k, const void* v, const int32_t* row_ptr,
                             const int32_t* col_idx, const int32_t* perm, const int32_t* seg_start,
                             const wa_shape* shape,
                             float softmax_scale, int32_t n_xcd, void* o, float* lse, int32_t* status,
                             void* workspace, size_t workspace_bytes, void* stream) {
  Dims d;
  wa_status s = check_shape(shape, &d);
  if (s != WA_OK) return s;
  s = check_attn_common(q, k, v, o, n_xcd, lse, status);
  if (s != WA_OK) return s;
  if (!row_ptr || !col_idx) return fail(WA_ERR_INVALID_ARG, "row_ptr and col_idx must be non-null");
  s = check_ws(workspace, workspace_bytes, attn_csr_ws_bytes(d));
  if (s != WA_OK) return s;
  s = launch_attn(q, k, v, nullptr, workspace, row_ptr, col_idx, perm, seg_start, d, softmax_scale, n_xcd, 0, o, lse,
                  status, (hipStream_t)stream);
  if (s != WA_OK) return s;
  return ok();
}

wa_status wa_sparse_attn_vt_noalloc(const void* q, const void* k, const void* vt, const int32_t* row_ptr,
                                    const int32_t* col_idx, const int32_t* perm, const int32_t* seg_start,
                                    const wa_shape* shape, const wa_attn_options* options, void* o, float* lse,
                                    int32_t* status, void* stream) {
  Dims d;
  wa_status s = check_shape(shape, &d);
  if (s != WA_OK) return s;
  if (!options) return fail(WA_ERR_INVALID_ARG, "options is null");
  s = check_attn_common(q, k, vt, o, options->n_xcd, lse, status);
  if (s != WA_OK) return s;
  if (options->head_order != WA_HEADS_IN_ORDER && options->head_order != WA_HEADS_INTERLEAVED)
    return fail(WA_ERR_INVALID_ARG, "head_order %d invalid", options->head_order);
  if (!row_ptr || !col_idx) return fail(WA_ERR_INVALID_ARG, "row_ptr and col_idx must be non-null");
  // the kernels index the scheduler state with the call's own n_xcd
  const size_t need = wa::sched_state_ints(d.bh, d.mb, options->n_xcd) * 4;
  if (need > (size_t)WA_NOALLOC_SCRATCH_BYTES)
    return fail(WA_ERR_WORKSPACE,
                "scheduler state of %zu bytes (batch*heads %lld, M_B %d, n_xcd %d) exceeds the %d-byte static scratch",
                need, (long long)d.bh, d.mb, options->n_xcd, WA_NOALLOC_SCRATCH_BYTES);
  int32_t* scratch = nullptr;
  size_t have = 0;
  hipError_t e = wa_noalloc_scratch(&scratch, &have);
  if (e != hipSuccess) return hip_fail(e, "static scratch lookup");
  if (need > have) return fail(WA_ERR_WORKSPACE, "static scratch holds %zu bytes, %zu needed", have, need);
  s = launch_attn(q, k, nullptr, vt, scratch, row_ptr, col_idx, perm, seg_start, d, options->softmax_scale,
                  options->n_xcd, options->head_order, o, lse, status, (hipStream_t)stream);
  if (s != WA_OK) return s;
  return ok();
}

wa_status wa_transpose_v(const void* v, const wa_shape* shape, void* vt, void* stream) {
  Dims d;
  wa_status s = check_shape(shape, &d);
  if (s != WA_OK) return s;
  if (!v || !vt) return fail(WA_ERR_INVALID_ARG, "v and vt must be non-null");
  if (!aligned(v, 16) || !aligned(vt, 16)) return fail(WA_ERR_ALIGNMENT, "v and vt must be 16-byte aligned");
  hipError_t e = wa_launch_transpose_v(v, vt, d.bh, d.n, d.mb, d.d, d.blk, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "transpose launch");
  return ok();
}

wa_status wa_attn_vt_workspace_size(const wa_shape* shape, size_t* bytes) {
  Dims d;
  wa_status s = check_shape(shape, &d);
  if (s != WA_OK) return s;
  if (!bytes) return fail(WA_ERR_INVALID_ARG, "bytes is null");
  *bytes = attn_sched_bytes(d);
  return ok();
}

wa_status wa_sparse_attn_vt(const void* q, const void* k, const void* vt, const int32_t* row_ptr,
                            const int32_t* col_idx, const int32_t* perm, const int32_t* seg_start,
                            const wa_shape* shape, const wa_attn_options* options, void* o, float* lse,
                            int32_t* status, void* workspace, size_t workspace_bytes, void* stream) {
  Dims d;
  wa_status s = check_shape(shape, &d);
  if (s != WA_OK) return s;
  if (!options) return fail(WA_ERR_INVALID_ARG, "options is null");
  s = check_attn_common(q, k, vt, o, options->n_xcd, lse, status);
  if (s != WA_OK) return s;
  if (options->head_order != WA_HEADS_IN_ORDER && options->head_order != WA_HEADS_INTERLEAVED)
    return fail(WA_ERR_INVALID_ARG, "head_order %d invalid", options->head_order);
  if (!row_ptr || !col_idx) return fail(WA_ERR_INVALID_ARG, "row_ptr and col_idx must be non-null");
  s = check_ws(workspace, workspace_bytes, attn_sched_bytes(d));
  if (s != WA_OK) return s;
  s = launch_attn(q, k, nullptr, vt, workspace, row_ptr, col_idx, perm, seg_start, d, options->softmax_scale,
                  options->n_xcd, options->head_order, o, lse, status, (hipStream_t)stream);
  if (s != WA_OK) return s;
  return ok();
}

/* Diagnostic: evaluates on the GPU the fp64 operations the exact permutation relies on
 * (sqrt, division, int64 -> fp64, rint, uncontracted multiply-subtract, ldexp) so they can be
 * compared bit for bit with IEEE results on the host. a, b: double [n]; c: int64 [n];
 * out: double [n][6]. Device pointers. */
wa_status wa_fp64_probe(const double* a, const double* b, const int64_t* c, double* out, int32_t n, void* stream) {
  if (!a || !b || !c || !out) return fail(WA_ERR_INVALID_ARG, "null pointer");
  if (n < 0) return fail(WA_ERR_INVALID_ARG, "n < 0");
  hipError_t e = wa_launch_fp64_probe(a, b, c, out, n, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "fp64 probe launch");
  return ok();
}

wa_status wa_xcc_probe(int32_t* out, int32_t n_wg, void* stream) {
  if (!out) return fail(WA_ERR_INVALID_ARG, "out is null");
  if (n_wg < 0) return fail(WA_ERR_INVALID_ARG, "n_wg < 0");
  hipError_t e = wa_launch_xcc_probe(out, n_wg, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "xcc probe launch");
  return ok();
}

}  // extern "C"
