// Host scheduling policy of the attention path: the token-budget steps of a
// chunked prefill and the split point of the shared-prefix (cascade) pass.
//
// Chunked prefill is how a serving engine bounds the new tokens of one
// scheduler step (InferLog section 3.3 tunes that bound, vLLM's
// max-num-batched-tokens; section 4.1's PC-Chunk baseline runs prefix caching
// with it).  The cascade split is the prefix every prompt of a batch shares
// (the instruction and leading demonstrations, section 2.1.1), which the
// prefix cache stores once (section 2.1.2).
#include <cstdint>

#include "../../include/ilpc.h"
#include "ilpc_internal.h"

using ilpc::set_error;

extern "C" int ilpc_chunk_schedule(const int32_t* q_lens, int32_t B, int32_t budget, int32_t max_pieces,
                                   int32_t* piece_req, int32_t* piece_off, int32_t* piece_len,
                                   int32_t* piece_step, int32_t* n_pieces, int32_t* n_steps) {
  static const char* fn = "ilpc_chunk_schedule";
  if (!n_pieces || !n_steps) return set_error(ILPC_EINVAL, "%s: n_pieces / n_steps is NULL", fn);
  *n_pieces = 0;
  *n_steps = 0;
  if (B < 0 || budget < 1 || max_pieces < 0)
    return set_error(ILPC_EINVAL, "%s: B %d, budget %d, max_pieces %d", fn, B, budget, max_pieces);
  if (B > 0 && !q_lens) return set_error(ILPC_EINVAL, "%s: q_lens is NULL", fn);
  // Count first: pieces and steps, with every length checked.
  int64_t total = 0, pieces = 0, room = budget;
  for (int32_t r = 0; r < B; ++r) {
    const int64_t n = q_lens[r];
    if (n < 0) return set_error(ILPC_EINVAL, "%s: q_lens[%d] = %lld < 0", fn, r, (long long)n);
    // A request of n tokens starting with `room` left in the current step
    // spans 1 + ceil(max(0, n - room) / budget) pieces.
    if (n > 0) {
      pieces += 1 + (n > room ? (n - room + budget - 1) / budget : 0);
      const int64_t used = (budget - room + n) % budget;
      room = used == 0 ? budget : budget - used;
    }
    total += n;
  }
  const int64_t steps = (total + budget - 1) / budget;
  if (pieces > INT32_MAX || steps > INT32_MAX) return set_error(ILPC_EUNSUP, "%s: schedule too long", fn);
  *n_pieces = int32_t(pieces);
  *n_steps = int32_t(steps);
  if (pieces > max_pieces)
    return set_error(ILPC_EINVAL, "%s: %lld pieces do not fit in %d", fn, (long long)pieces, max_pieces);
  if (pieces > 0 && (!piece_req || !piece_off || !piece_len || !piece_step))
    return set_error(ILPC_EINVAL, "%s: a piece output is NULL", fn);
  // First come, first served: a step takes what is left of the current
  // request, then the following requests, and cuts the last one it reaches.
  int32_t k = 0, step = 0;
  room = budget;
  for (int32_t r = 0; r < B; ++r) {
    int64_t off = 0;
    while (off < q_lens[r]) {
      const int64_t take = q_lens[r] - off < room ? q_lens[r] - off : room;
      piece_req[k] = r;
      piece_off[k] = int32_t(off);
      piece_len[k] = int32_t(take);
      piece_step[k] = step;
      ++k;
      off += take;
      room -= take;
      if (room == 0) {
        ++step;
        room = budget;
      }
    }
  }
  return ILPC_OK;
}

extern "C" int ilpc_shared_prefix_len(const int32_t* cached_len, const int32_t* block_tables, int32_t B,
                                      int32_t max_blocks, int32_t* shared_len) {
  static const char* fn = "ilpc_shared_prefix_len";
  if (!shared_len) return set_error(ILPC_EINVAL, "%s: shared_len is NULL", fn);
  *shared_len = 0;
  if (B < 0 || max_blocks < 1) return set_error(ILPC_EINVAL, "%s: B %d, max_blocks %d", fn, B, max_blocks);
  if (B == 0) return ILPC_OK;
  if (!cached_len || !block_tables) return set_error(ILPC_EINVAL, "%s: NULL pointer", fn);
  int32_t min_cached = cached_len[0];
  for (int32_t r = 0; r < B; ++r) {
    if (cached_len[r] < 0) return set_error(ILPC_EINVAL, "%s: cached_len[%d] < 0", fn, r);
    if (cached_len[r] < min_cached) min_cached = cached_len[r];
  }
  int64_t n = min_cached / 16;
  if (n > max_blocks) n = max_blocks;
  int64_t run = 0;
  for (; run < n; ++run) {
    const int32_t id = block_tables[run];
    if (id < 0) break;
    bool same = true;
    for (int32_t r = 1; r < B && same; ++r) same = block_tables[int64_t(r) * max_blocks + run] == id;
    if (!same) break;
  }
  *shared_len = int32_t(run * 16);
  return ILPC_OK;
}

// Measured on MI355X against the single pass: sweep100's prefill (976 shared
// keys, 48 own) 9% faster in one launch; sweep75 (736 shared, 288 own) 3%
// slower; llama8b and qwen7b (256 / 512 shared, 300-700 own) 9-12% slower.
// The split removes no matrix-core work; it pays only where the shared keys
// dominate and each request's own keys past them fit in two 64-key tiles.
// Decode-shaped batches (at most 32 query columns per request and kv head)
// keep the single pass: the decode kernel reads a shared prefix from L2 per
// request (sweep100's decode steps: 47 us single, 72 us split).
extern "C" int ilpc_prefer_shared_split(const int32_t* seq_lens, int32_t B, int32_t max_q_len, int32_t Hq,
                                        int32_t Hkv, int32_t shared_len, int32_t* use) {
  static const char* fn = "ilpc_prefer_shared_split";
  if (!use) return set_error(ILPC_EINVAL, "%s: use is NULL", fn);
  *use = 0;
  if (B < 0 || shared_len < 0 || max_q_len < 0 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0)
    return set_error(ILPC_EINVAL, "%s: B %d, shared_len %d, max_q_len %d, heads %d/%d", fn, B, shared_len,
                     max_q_len, Hq, Hkv);
  if (B == 0) return ILPC_OK;
  if (!seq_lens) return set_error(ILPC_EINVAL, "%s: seq_lens is NULL", fn);
  int32_t own_max = 0;
  for (int32_t r = 0; r < B; ++r) {
    if (seq_lens[r] < shared_len) return set_error(ILPC_EINVAL, "%s: seq_lens[%d] < shared_len", fn, r);
    own_max = seq_lens[r] - shared_len > own_max ? seq_lens[r] - shared_len : own_max;
  }
  const bool prefill_shaped = int64_t(max_q_len) * (Hq / Hkv) > 32;
  *use = prefill_shaped && shared_len >= 3 * 64 && own_max <= 2 * 64 ? 1 : 0;
  return ILPC_OK;
}
