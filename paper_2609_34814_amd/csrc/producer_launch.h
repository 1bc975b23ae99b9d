// Internal launch interface of the mask-producer kernels (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

struct WaProducerLaunch {
  const void* q;      // bf16 [bh][seq_len][head_dim]
  const void* k;
  float* means;       // workspace float32 [2][bh][mb][head_dim]: block means of Q, then K
  uint32_t* amax;     // workspace [2][bh]: bits of the per-head maximum |mean|
  uint32_t* bmax;     // workspace [2][bh][mb]: bits of each block's maximum |mean|
  int8_t* codes;      // [2][bh][mb][head_dim]: int8 codes of Q, then K
  uint8_t* mask;      // out [bh][mb][mb]
  uint32_t* queue;    // workspace [wa_producer_queue_words(bh)]: the work queue and its flags
  int32_t* status;    // out, nullable: WA_PRODUCE_WAIT_EXPIRED
  int32_t bh, mb, seq_len, block, head_dim, keep, diagonal;
};

// 32-bit words of the producer's work queue: two counters, padding, then per (tensor, head) the
// blocks pooled and a codes-written flag.
inline int64_t wa_producer_queue_words(int64_t bh) { return 64 + 4 * bh; }

hipError_t wa_launch_producer(const WaProducerLaunch& a, hipStream_t stream);
