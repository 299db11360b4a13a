// Internal helpers shared by the library's translation units (not part of the ABI).
#pragma once

#include <cstdarg>
#include <cstddef>
#include <cstdint>

namespace ilpc {

// Records a message for ilpc_last_error() on the calling thread and returns `code`.
int set_error(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

// Decode-shaped paged attention (at most 32 query columns, q_len * Hq / Hkv,
// per request): one wave per (request, kv head).  Arguments as for
// ilpc_paged_prefill_attn, already checked; scale_log2 = softmax scale *
// log2(e); stream is a hipStream_t.
// With 1 < n_split <= kMaxSplit each pair's keys are cut into n_split
// ranges, one wave each, whose partial states go to `part`
// (decode_split_bytes() bytes, 16-byte aligned) and are merged by a second
// launch.
int launch_decode_attn(const uint16_t* q, const uint16_t* k_pool, const uint16_t* v_pool, int num_blocks,
                       const int32_t* block_tables, int max_blocks, const int32_t* cu_q,
                       const int32_t* seq_lens, int B, int max_q_len, int Hq, int Hkv, int D,
                       float scale_log2, uint16_t* out, int n_split, float* part, void* stream);
size_t decode_split_bytes(int B, int max_q_len, int Hq, int Hkv, int D, int n_split);
constexpr int kMaxSplit = 64;

}  // namespace ilpc
