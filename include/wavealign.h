/*
 * wavealign.h - C ABI of the MI355X (gfx950) block-sparse attention path with
 * cache-aware query-row reordering (WaveAlign, arXiv 2609.34814).
 *
 * Two operations follow the paper's problem statement:
 *   - wa_build_permutation: block mask M_h in {0,1}^{M_B x N_B} per head in,
 *     row permutation P_h out (Sec. IV-B, Eq. 1; Alg. 1 and Alg. 2; the
 *     adaptive skip of Sec. IV-E);
 *   - wa_sparse_attn: Q, K, V and M in, O out in the original row order
 *     (Sec. II-B, II-C: FlashAttention-style query-block outer loop over the
 *     mask-selected KV blocks; Sec. IV-A: only the execution order changes).
 *
 * Conventions (all entry points)
 *   - Tensor and mask pointers are DEVICE pointers owned by the caller.
 *     Scalar parameter structs are HOST pointers, read during the call only.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = the default stream)
 *     and is asynchronous: no entry point synchronises (except the debugging
 *     check wa_check_perm), allocates device memory or frees caller memory. Scratch memory comes from the caller's
 *     `workspace` (device memory, 256-byte aligned, of at least the size the
 *     matching *_workspace_size call reports).
 *   - Every argument is validated before anything is enqueued; on error the
 *     call returns a negative wa_status, enqueues nothing and leaves all
 *     outputs untouched. wa_last_error() then describes the failure
 *     (thread-local, valid until the thread's next call). WA_ERR_HIP means a
 *     HIP runtime call or a launch failed after validation.
 *   - No C++ exception crosses the ABI.
 *   - Shapes: Q, K, V, O are bf16 [batch][heads][seq_len][head_dim],
 *     contiguous. Blocks are runs of `block` consecutive tokens; block j holds
 *     tokens [j*block, min((j+1)*block, seq_len)), so M_B = N_B =
 *     ceil(seq_len / block) and the last block may be ragged. The mask is
 *     uint8 [batch][heads][M_B][N_B], row-major; nonzero = the query block
 *     attends to the KV block.
 *   - Supported: head_dim in {64, 128}; block in {64, 128}; 1 <= M_B <= 4096;
 *     batch*heads*M_B*N_B < 2^31.
 *   - perm[b][h][s] is the original query block executed at slot s (row s of
 *     P_h M_h, Eq. 1). Each perm[b][h] must be a permutation of 0..M_B-1.
 */
#ifndef WAVEALIGN_H
#define WAVEALIGN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define WA_ABI_VERSION 3
#define WA_MAX_BLOCKS 4096

typedef enum wa_status {
  WA_OK = 0,
  WA_ERR_INVALID_ARG = -1,  /* null pointer, non-positive size, bad enum value */
  WA_ERR_UNSUPPORTED = -2,  /* head_dim / block / size outside the supported set */
  WA_ERR_ALIGNMENT = -3,    /* tensor not 16-byte aligned, workspace not 256-byte aligned */
  WA_ERR_WORKSPACE = -4,    /* workspace smaller than required */
  WA_ERR_INVALID_PERM = -5, /* wa_check_perm: some perm[b][h] is not a permutation of 0..M_B-1 */
  WA_ERR_HIP = -6           /* a HIP runtime call or kernel launch failed */
} wa_status;

typedef struct wa_shape {
  int32_t batch;
  int32_t heads;
  int32_t seq_len;   /* tokens N */
  int32_t head_dim;  /* d */
  int32_t block;     /* tokens per query / KV block */
} wa_shape;

/* Offline-profile constants of the adaptive skip (Sec. IV-E). A head keeps the
 * identity order when any case fires (skip_mode = WA_SKIP_AUTO):
 *   1  distinct_kv_blocks * kv_block_bytes <= cache_bytes             (fits in cache)
 *   2  nnz * gain_ns_per_block < ovh_ns_fixed + ovh_ns_per_row * M_B
 *                                 + ovh_ns_per_nnz * nnz                (too little work)
 *      with the ovh_fused_* constants instead when M_B <= fused_max_blocks (heads the
 *      permutation builds in one workgroup, whose cost grows differently)
 *   3  sum_i |M_i & M_i+1| / sum_i |M_i | M_i+1| >= j_max              (already local)
 *      or, once the order P is built, J(P) <= J(natural order), with J that
 *      overlap over consecutive rows of an order, compared as exact integer
 *      cross-products                                                    (no locality gained)
 *   4  (lambda_1 + lambda_2) / ||M~||_F^2 < eta_min                      (no rank-2 structure)
 * Each comparison is one fixed sequence of IEEE fp64 operations. */
typedef struct wa_skip_profile {
  double cache_bytes;
  double gain_ns_per_block;
  double ovh_ns_fixed;
  double ovh_ns_per_row;
  double ovh_ns_per_nnz;
  double j_max;
  double eta_min;
  double fused_max_blocks;
  double ovh_fused_ns_fixed;
  double ovh_fused_ns_per_row;
  double ovh_fused_ns_per_nnz;
} wa_skip_profile;

enum { WA_SKIP_AUTO = 0, WA_SKIP_NEVER = 1, WA_SKIP_ALWAYS = 2 };

/* head_flags bits written by wa_build_permutation */
enum {
  WA_FLAG_FITS_CACHE = 1,
  WA_FLAG_LITTLE_WORK = 2,
  WA_FLAG_LOCAL = 4,
  WA_FLAG_UNSTRUCTURED = 8,
  WA_FLAG_DEGENERATE = 16,  /* centred mask has no direction; Stage 1 kept the identity order */
  WA_FLAG_IDENTITY = 64     /* the identity permutation was returned */
};

typedef struct wa_perm_params {
  int32_t wave_per_xcd;  /* W: resident query-block tasks per XCD; 0 = wa_wave_size() for the shape */
  int32_t n_xcd;         /* contiguous segments, one per XCD (8 on MI355X); 1 = Alg. 2 as printed */
  int32_t iters;         /* T subspace iterations (Alg. 1), 1..64; the paper uses 5-15 */
  int32_t skip_mode;     /* WA_SKIP_AUTO / WA_SKIP_NEVER / WA_SKIP_ALWAYS */
  uint64_t seed;         /* SplitMix64 counter base of the random start block */
  const wa_skip_profile* profile;  /* host pointer; NULL = wa_default_skip_profile() */
} wa_perm_params;

/* Library version (WA_ABI_VERSION). */
int32_t wa_abi_version(void);

/* Static description of a status code. */
const char* wa_status_string(wa_status status);

/* Detail of the calling thread's last failed call ("" if none). */
const char* wa_last_error(void);

/* Built-in skip-profile constants. */
wa_status wa_default_skip_profile(wa_skip_profile* out);

/* Query blocks resident per XCD for the attention kernel of this head_dim and
 * block (32 CUs per XCD x workgroups per CU). Queries the current device. */
wa_status wa_wave_size(int32_t head_dim, int32_t block, int32_t* wave_per_xcd);

/* Per-head mask statistics (Sec. II-B row NNZ n_i; Alg. 1 column counts c = M^T 1;
 * the inputs of the skip rule of Sec. IV-E).
 *   row_nnz    out int32 [B][H][M_B]
 *   col_cnt    out int32 [B][H][N_B]
 *   head_stats out int64 [B][H][6]: nnz, distinct columns, sum_i |M_i & M_i+1|,
 *              sum_i |M_i | M_i+1|, sum_j c_j^2, 0
 *   workspace  >= wa_perm_workspace_size(shape). */
wa_status wa_mask_stats(const uint8_t* mask, const wa_shape* shape, int32_t* row_nnz, int32_t* col_cnt,
                        int64_t* head_stats, void* workspace, size_t workspace_bytes, void* stream);

/* Workspace bytes needed by wa_build_permutation and wa_mask_stats: the bit-packed
 * rows and columns of the mask, per-head statistics, and the state of the subspace
 * iteration (X and the two centred products), about B*H*M_B*(2*ceil(N_B/64)*8 + 48)
 * bytes.
 * Calls that share a workspace must not overlap. */
wa_status wa_perm_workspace_size(const wa_shape* shape, size_t* bytes);

/* Two-stage cache-aware row permutation per head (Alg. 2 with MFCSI, Alg. 1):
 * Stage 1 orders rows by the polar angle of their rank-2 centred spectral
 * embedding (Eq. 2-4); the order is split into n_xcd contiguous segments of
 * equal work (sum of n_i + 1), one per XCD, and each segment into buckets of
 * wave_per_xcd rows; Stage 2 sorts each bucket by descending n_i (stable).
 * Integer-exact fixed-point arithmetic makes the result identical on every run
 * and to the reference reading.
 *   perm         out int32 [B][H][M_B] (required)
 *   seg_start    out int32 [B][H][n_xcd+1] slot where each XCD segment starts
 *                (last entry M_B), nullable; pass it to wa_sparse_attn with the same n_xcd
 *   head_flags   out uint8 [B][H] WA_FLAG_* bits, nullable
 *   embedding    out int32 [B][H][M_B][2] canonical (u1, u2), 2^30 per unit, nullable
 *                (zeros for heads that skipped Stage 1)
 *   stage1_order out int32 [B][H][M_B] Stage-1 order, nullable (identity when skipped) */
wa_status wa_build_permutation(const uint8_t* mask, const wa_shape* shape, const wa_perm_params* params,
                               int32_t* perm, int32_t* seg_start, uint8_t* head_flags, int32_t* embedding,
                               int32_t* stage1_order, void* workspace, size_t workspace_bytes, void* stream);

/* Debugging check of a permutation argument (Sec. IV-B: P_h is a permutation
 * matrix): every perm[b][h] must hold each of 0..M_B-1 exactly once.
 *   perm       int32 [B][H][M_B], device
 *   head_ok    out int32 [B][H], device, nullable: 1 where the head's order is a
 *              permutation, else 0
 *   workspace  >= wa_check_perm_workspace_size(shape), 256-byte aligned
 * Unlike every other entry point this call SYNCHRONISES `stream` (it copies the
 * count of bad heads to the host) and returns WA_ERR_INVALID_PERM when any head
 * fails, WA_OK otherwise. */
wa_status wa_check_perm(const int32_t* perm, const wa_shape* shape, int32_t* head_ok, void* workspace,
                        size_t workspace_bytes, void* stream);
wa_status wa_check_perm_workspace_size(const wa_shape* shape, size_t* bytes);

/* Compacted per-row KV-block index lists (the mask-selected inner loop of Sec. II-C):
 *   row_ptr out int32 [B][H][M_B+1]: exclusive prefix sum of n_i, local to the head
 *   col_idx out int32, capacity B*H*M_B*N_B: head (b,h)'s list starts at
 *           (b*H+h)*M_B*N_B; row i's indices are ascending j with M[i][j] != 0. */
wa_status wa_compact_mask(const uint8_t* mask, const wa_shape* shape, int32_t* row_ptr, int32_t* col_idx,
                          void* stream);

/* Status word of wa_produce_block_mask (device int32, nullable): zeroed by the call; bit 1
 * is set if a selection item's wait for the codes of its head ran out. The call takes its
 * items from a queue in which every such wait depends only on items taken earlier by running
 * workgroups that never wait, so the bit cannot be set; if it were, the mask is not valid.
 * Readable once the stream has passed the call. */
enum { WA_PRODUCE_WAIT_EXPIRED = 1 };

/* Pooled-score top-k block mask: a content-dependent producer of the mask the path
 * consumes (Sec. II-B: dynamic sparse attention predicts block relevance from pooled
 * Q/K features). Per head:
 *   qbar_i = mean of the Q rows of block i (ascending float32 fold, then one
 *            correctly rounded division by the block's token count); kbar_j alike;
 *   codes  = rint(mean * fl32(127 / max_head |mean|)), clamped to [-127, 127]
 *            (all zero when the maximum is 0), for Q and K separately;
 *   s_ij   = sum_c qcode_i[c] * kcode_j[c] (exact integer);
 *   row i keeps its `keep` largest s_ij (equal scores: smaller j first) and, if
 *   `diagonal` is nonzero, block j = i.
 *   q, k      bf16 [B][H][N][d], device
 *   keep      >= 0; values >= N_B keep every block
 *   mask      out uint8 [B][H][M_B][N_B], 1 = kept
 *   codes     out int8 [2][B][H][M_B][d] (Q codes, then K codes), nullable
 *   status    out int32 device word (WA_PRODUCE_WAIT_EXPIRED), nullable, 4-byte aligned
 *   workspace >= wa_mask_producer_workspace_size(shape), 256-byte aligned. */
wa_status wa_produce_block_mask(const void* q, const void* k, const wa_shape* shape, int32_t keep, int32_t diagonal,
                                uint8_t* mask, int8_t* codes, int32_t* status, void* workspace,
                                size_t workspace_bytes, void* stream);

/* Workspace bytes needed by wa_produce_block_mask: float32 block means, per-block and
 * per-head maxima of Q and K, their int8 codes, and the call's work queue (64 + 4*B*H
 * uint32 counters and flags, cleared by the call itself). Calls that share a workspace
 * must not overlap. */
wa_status wa_mask_producer_workspace_size(const wa_shape* shape, size_t* bytes);

/* Workspace bytes needed by wa_sparse_attn: the scheduler state (queue counters,
 * per-queue prefix tables and the per-queue order of the last heads: 64 + 64 * (B*H + 1)
 * int32 rounded up to 64 entries, plus 64 * T * M_B int32 with T = min(B*H, 16384 / M_B, 256)
 * rounded up to 64 entries, plus 64 + B*H*M_B int32 for the head-interleaved order,
 * rounded up to 256 bytes),
 * a zero-padded transposed copy of V (bf16 [B][H][head_dim][M_B*block], rounded up
 * to 256 bytes), then the compacted lists. The first two parts (the leading part)
 * suffice for wa_sparse_attn_csr. Calls that share a workspace must not overlap. */
wa_status wa_attn_workspace_size(const wa_shape* shape, size_t* bytes);

/* Status word of the attention calls (device int32, nullable): zeroed by the call, then
 * bits are set for what the call found. An invalid perm entry (outside 0..M_B-1)
 * occupies its slot without computing anything, so the query block it should have
 * named keeps whatever O held; an invalid KV index (outside 0..N_B-1, only possible
 * with caller-built lists) is read as block 0. Readable once the stream has passed
 * the call. Bijectivity of perm is not checked here (wa_check_perm does). */
enum { WA_ATTN_BAD_PERM = 1, WA_ATTN_BAD_KV_INDEX = 2 };

/* Block-sparse attention forward: for every query block i and token q in it,
 * O_q = softmax(scale * Q_q K_S^T) V_S over the tokens of the KV blocks with
 * M[i][j] != 0, visited in ascending j (Sec. II-B, II-C). bf16 inputs, fp32
 * accumulation, bf16 output. Query block i runs at the slot s with perm[s] = i
 * and is read and written at its original rows (the inverse permutation of
 * Sec. IV-A is fused into the store), so O is identical for every perm.
 * A query block with no kept KV block gets O = 0 and LSE = -inf. The softmax
 * takes the scores of each row's first kept block as its reference maximum; a
 * row whose later scores exceed it by 32 or more (log2 units) is recomputed
 * against its exact maximum within the same call. Inputs must be finite.
 *   q, k, v      bf16 [B][H][N][d], 16-byte aligned
 *   perm         int32 [B][H][M_B], NULL = identity (not checked for bijectivity)
 *   seg_start    int32 [B][H][n_xcd+1] XCD segment table from wa_build_permutation,
 *                NULL = segments of equal row count (the first M_B mod n_xcd one longer)
 *   softmax_scale  <= 0 selects 1/sqrt(d)
 *   n_xcd        number of XCD segments, 1..64. The kernel is persistent (one workgroup
 *                per resident slot); queue x holds segment x of every head, heads in order,
 *                and a workgroup takes the next slot of the queue of the XCD it runs on
 *                (hardware XCC id mod n_xcd), then of the other queues once that one is
 *                empty. 1: one queue, plain slot order on every XCD. In the last
 *                T = min(B*H, 16384 / M_B, 256) heads of each queue, a slot whose row
 *                could still be running when the rest of the queue is done (twice its
 *                block count times the queue's share of workgroups exceeds the blocks
 *                queued after it) is taken first, longest first; the others keep their
 *                order. The order changes when rows run, never what they compute.
 *   o            out bf16 [B][H][N][d]
 *   lse          out float [B][H][N] natural-log sum-exp of the scaled scores, nullable
 *   status       out int32 status word (WA_ATTN_* bits), device, nullable
 *   workspace    >= wa_attn_workspace_size(shape) */
wa_status wa_sparse_attn(const void* q, const void* k, const void* v, const uint8_t* mask, const int32_t* perm,
                         const int32_t* seg_start, const wa_shape* shape, float softmax_scale, int32_t n_xcd,
                         void* o, float* lse, int32_t* status, void* workspace, size_t workspace_bytes,
                         void* stream);

/* As wa_sparse_attn, from lists already built by wa_compact_mask (row i of head
 * (b,h) visits col_idx[(b*H+h)*M_B*N_B + row_ptr[b][h][i] ...] in list order).
 * workspace >= the scheduler and V^T parts of wa_attn_workspace_size, 256-byte aligned. */
wa_status wa_sparse_attn_csr(const void* q, const void* k, const void* v, const int32_t* row_ptr,
                             const int32_t* col_idx, const int32_t* perm, const int32_t* seg_start,
                             const wa_shape* shape,
                             float softmax_scale, int32_t n_xcd, void* o, float* lse, int32_t* status,
                             void* workspace, size_t workspace_bytes, void* stream);

/* V in the layout the attention kernel reads its P V operand from (Sec. II-C: the
 * value tile of each kept KV block): vt[b][h][c][t] = V[b][h][t][c] for tokens
 * t < N and 0 for N <= t < M_B*block.
 *   v   bf16 [B][H][N][d], 16-byte aligned
 *   vt  out bf16 [B][H][d][M_B*block], 16-byte aligned
 * A model whose value projection writes this layout directly can skip this call and
 * hand its output to wa_sparse_attn_vt. */
wa_status wa_transpose_v(const void* v, const wa_shape* shape, void* vt, void* stream);

/* Order of the query-block tasks of different heads within each task queue.
 * IN_ORDER runs the heads one after another (each queue finishes head h's segment
 * before head h+1's), so one head's K/V is in use at a time, as in the paper's
 * sequential-head scheduling (Sec. V); INTERLEAVED deals the slots round-robin over the
 * heads (slot r of every head, then slot r+1), so query blocks of all heads run
 * together, as a head-parallel scheduler does (the baseline of Sec. VI-B). Both compute
 * the same O; only the IN_ORDER form applies the end-of-launch order of the last heads. */
enum { WA_HEADS_IN_ORDER = 0, WA_HEADS_INTERLEAVED = 1 };

typedef struct wa_attn_options {
  float softmax_scale;  /* <= 0 selects 1/sqrt(d) */
  int32_t n_xcd;        /* XCD segments / task queues, 1..64 (as for wa_sparse_attn) */
  int32_t head_order;   /* WA_HEADS_IN_ORDER or WA_HEADS_INTERLEAVED */
} wa_attn_options;

/* Workspace bytes needed by wa_sparse_attn_vt: the scheduler state of
 * wa_attn_workspace_size alone. */
wa_status wa_attn_vt_workspace_size(const wa_shape* shape, size_t* bytes);

/* As wa_sparse_attn_csr, with V already in the layout wa_transpose_v writes, so the
 * call reads V^T tiles straight from the caller's tensor (no copy of V per call).
 *   vt         bf16 [B][H][d][M_B*block], 16-byte aligned; entries of tokens >= N must
 *              be finite (wa_transpose_v writes zeros)
 *   options    host pointer: softmax scale, n_xcd, head order
 *   status     as for wa_sparse_attn
 *   workspace  >= wa_attn_vt_workspace_size(shape), 256-byte aligned */
wa_status wa_sparse_attn_vt(const void* q, const void* k, const void* vt, const int32_t* row_ptr,
                            const int32_t* col_idx, const int32_t* perm, const int32_t* seg_start,
                            const wa_shape* shape, const wa_attn_options* options, void* o, float* lse,
                            int32_t* status, void* workspace, size_t workspace_bytes, void* stream);

/* For callers that cannot allocate device memory: code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc. The same computation as
 * wa_sparse_attn_vt, with the scheduler state (queue counters, prefix tables, the
 * orders of the last heads and the head-interleaved table) kept in a static device
 * array of the library instead of a workspace: WA_NOALLOC_SCRATCH_BYTES per GPU,
 * taken when the library's code is loaded on that GPU and held until the process
 * ends. The call allocates and frees nothing. A shape whose state needs more
 * (64 + n_xcd*(B*H+1) rounded up to 64, + n_xcd*T*M_B rounded up to 64, + 64 + B*H*M_B
 * int32, T as for wa_attn_workspace_size) is rejected with WA_ERR_WORKSPACE before
 * anything is enqueued. Every call on one GPU uses that GPU's one array and rebuilds
 * it from scratch (counters are re-zeroed by a kernel, not a memset), so calls that
 * overlap on one GPU (two streams, or two host threads) race: the caller serialises
 * them. Arguments and status as for wa_sparse_attn_vt. */
#define WA_NOALLOC_SCRATCH_BYTES (4 * 1024 * 1024)
wa_status wa_sparse_attn_vt_noalloc(const void* q, const void* k, const void* vt, const int32_t* row_ptr,
                                    const int32_t* col_idx, const int32_t* perm, const int32_t* seg_start,
                                    const wa_shape* shape, const wa_attn_options* options, void* o, float* lse,
                                    int32_t* status, void* stream);

/* ---- diagnostics (used by the test suite; not needed by callers) ---- */

/* Evaluates on the GPU the fp64 operations the exact permutation relies on, for
 * comparison bit for bit with IEEE results on the host. Device pointers:
 * a, b double [n]; c int64 [n]; out double [n][6] =
 * { sqrt(|a|), a / b, (double)c, rint(a * 2^30), a*b - b*3 (two roundings, no
 * fused multiply-add), ldexp(a, (c & 31) - 16) }. */
wa_status wa_fp64_probe(const double* a, const double* b, const int64_t* c, double* out, int32_t n, void* stream);

/* Writes the XCD index each workgroup of an n_wg-workgroup grid ran on
 * (out: device int32 [n_wg]), to check the round-robin dispatch that the
 * XCD-aware slot mapping of wa_sparse_attn assumes. */
wa_status wa_xcc_probe(int32_t* out, int32_t n_wg, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* WAVEALIGN_H */
