// Paged K/V append and prefix-cached paged prefill attention for gfx950.
//
// InferLog (arXiv 2507.08523) section 2.1.2: with prefix caching only the
// cache-missing suffix of a prompt is prefilled; its queries attend to the
// reused KV of the cached prefix plus their own freshly stored KV (section
// 3.2.2).  This file holds the two device steps of that path:
//
//  * kv_append: scatter new K/V rows into 16-token pool blocks.  K blocks are
//    token-major [16][D]; V blocks are stored dimension-major [D][16] so the
//    attention kernel can feed them to the matrix cores without a transpose.
//  * paged_attn: causal grouped-query attention of the suffix queries.  A
//    work item is 256 query columns of one (request, kv head); a column is a
//    (token, q head of the group) pair, so the G heads of a group share every
//    K/V tile.  The kernel is persistent (one 8-wave workgroup per CU) and
//    takes items from per-XCD queues (with no more items than CUs, one item
//    per workgroup by position).  64-key tiles (4 pool blocks) stream
//    through a 4-tile ring in LDS, filled by direct global-to-LDS loads
//    issued a tile step ahead of use.  Per tile and wave:
//      S^T = K Q^T   on v_mfma_f32_32x32x16_bf16 (a lane owns one column),
//      causal mask, online softmax in fp32 on exp2 with the scale folded in:
//      the exponentials are taken against the running column max, and the
//      tile's column max is computed (and O rescaled) only when a lane's sum
//      of them leaves [0, 2^8] -- on an item's first tile, or when the max
//      has grown by several powers of two --,
//      O^T += V^T P^T on the same MFMA, P taken straight from the S^T
//      accumulators (K rows are staged in a permuted order that makes the
//      accumulator layout of S^T equal the operand layout P^T needs).
//    The two waves sharing a SIMD run these steps half a tile apart, so one
//    feeds the matrix core while the other computes the softmax.
//  * the same attention split at a prefix every request of the batch shares
//    (modes kShared / kSuffix: two launches; kFused: one launch whose items
//    are 256 columns of the whole batch, over the shared tiles and then each
//    of their requests' own tiles).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <climits>
#include <cstdint>
#include <type_traits>

#include "../../include/ilpc.h"
#include "ilpc_internal.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 16;                    // tokens per pool block
constexpr int kWaves = 8;                     // waves per attention workgroup
constexpr int kThreads = 64 * kWaves;
constexpr int kColsPerWave = 32;              // query columns per wave (MFMA N)
constexpr int kCols = kColsPerWave * kWaves;  // query columns per workgroup
constexpr int kKeys = 64;                     // keys per tile
constexpr int kTileBlocks = kKeys / kBlock;
constexpr int kStages = 4;                    // K/V tiles resident in the LDS ring
constexpr int kMaxGroup = 64;                 // largest Hq / Hkv accepted
constexpr int kDecodeCols = 32;               // query columns the decode kernel takes per request

// LDS row that holds tile key k.  Inside every 16 keys the groups [4,8) and
// [8,12) trade places, so that MFMA row m of S^T carries key sigma(m) and the
// fp32 accumulator registers of S^T line up with the bf16 operand of P^T:
// lane half h then holds keys 16c + 8h + 0..7 in registers 8c..8c+7.
__device__ __forceinline__ int key_row(int k) {
  const int grp = (k >> 2) & 3;
  return k + (grp == 1 ? 4 : (grp == 2 ? -4 : 0));
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// 16-byte slot of chunk c in LDS K row m: XOR-swizzled so that the 16 lanes an
// LDS cycle serves (16 consecutive rows, one chunk each) hit distinct banks.
template <int D>
__device__ __forceinline__ int k_slot(int m, int c) {
  return D == 128 ? (c ^ (m & 15)) : (c ^ ((m >> 1) & 7));
}

// 16-byte half (keys 0-7 or 8-15) of V row d of a [D][16] block in LDS.
__device__ __forceinline__ int v_slot(int d, int hf) { return hf ^ ((d >> 2) & 1) ^ ((d >> 3) & 1); }

// 16 bytes per lane from global memory straight into LDS at lds + 16 * lane
// (lds wave-uniform).  Issued as inline assembly so that the compiler does
// not track it: tracked, every LDS read would first wait for all such loads
// in flight, which defeats the multi-tile prefetch.  Callers wait with an
// explicit vmcnt.  M0 carries the LDS address; no other code in these
// kernels uses M0, so it is clobbered without being restored.  Kept out of
// the kernel templates: an LDS address-space cast instantiated in their
// host-side pass would drop the launch stubs.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void global_to_lds16(const void* src, uint8_t* lds) {
  const uint32_t lds_off = static_cast<uint32_t>(
      reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) uint8_t*)lds));
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(src), "s"(lds_off)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// max(x, x of the lane 32 apart): v_permlane32_swap exchanges the two wave halves.
__device__ __forceinline__ float max_across_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// ---------------------------------------------------------------------------
// kv_append: one workgroup per (logical block touched, kv head, request).
template <int D>
__global__ __launch_bounds__(256) void kv_append_kernel(
    const uint16_t* __restrict__ k_new, const uint16_t* __restrict__ v_new,
    uint16_t* __restrict__ k_pool, uint16_t* __restrict__ v_pool, int num_blocks,
    const int32_t* __restrict__ block_tables, int max_blocks, const int32_t* __restrict__ cu_new,
    const int32_t* __restrict__ start_pos, int max_new, int Hkv) {
  constexpr int kChunks = D / 8;  // 16-byte chunks per row
  __shared__ __attribute__((aligned(16))) uint16_t sv[kBlock][D + 8];
  const int r = blockIdx.z, h = blockIdx.y;
  const int row0 = cu_new[r];
  int n = cu_new[r + 1] - row0;
  if (n > max_new) n = max_new;
  const int start = start_pos[r];
  if (n <= 0 || start < 0) return;
  const int lb = start / kBlock + int(blockIdx.x);
  const int p0 = max(start, lb * kBlock), p1 = min(start + n, (lb + 1) * kBlock);
  if (p0 >= p1 || lb >= max_blocks) return;
  const int phys = block_tables[size_t(r) * max_blocks + lb];
  if (phys < 0 || phys >= num_blocks) return;
  const int tid = threadIdx.x;
  const size_t kblk = (size_t(phys) * Hkv + h) * kBlock * D;  // same offset for K and V blocks

  for (int idx = tid; idx < kBlock * kChunks; idx += 256) {
    const int slot = idx / kChunks, c = idx % kChunks;
    const int p = lb * kBlock + slot;
    if (p >= p0 && p < p1) {
      const size_t src = (size_t(row0 + p - start) * Hkv + h) * D + c * 8;
      *(u32x4*)(k_pool + kblk + size_t(slot) * D + c * 8) = *(const u32x4*)(k_new + src);
      *(u32x4*)(&sv[slot][c * 8]) = *(const u32x4*)(v_new + src);
    }
  }
  __syncthreads();
  for (int idx = tid; idx < 2 * D; idx += 256) {
    const int d = idx >> 1, hf = idx & 1;
    const int pb = lb * kBlock + hf * 8;
    uint16_t* dst = v_pool + kblk + size_t(d) * kBlock + hf * 8;
    if (pb >= p0 && pb + 8 <= p1) {
      u32x4 w;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        w[e] = uint32_t(sv[hf * 8 + 2 * e][d]) | (uint32_t(sv[hf * 8 + 2 * e + 1][d]) << 16);
      *(u32x4*)dst = w;
    } else {
      for (int e = 0; e < 8; ++e) {
        const int p = pb + e;
        if (p >= p0 && p < p1) dst[e] = sv[hf * 8 + e][d];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// paged attention.  Work items are (column tile, kv head, request) triples,
// numbered request-major with the heaviest column tile of a (request, kv head)
// first.  The kernel is persistent: one workgroup per CU takes items from
// eight queues, one per XCD, each holding a contiguous range of item numbers
// so that the items sharing one (request, kv head) -- and so the same K/V
// blocks -- are worked on under one XCD's L2.  A workgroup drains the queue
// of its own XCD first, then helps the others.  The queue counters live in
// the caller's workspace; the last workgroup to finish clears them again.
//
// K/V tiles stream through a ring of kStages tiles in LDS, filled straight
// from HBM by global_load_lds (tile j+2 issued while tile j's softmax runs).
// Each wave loads one
// pool block (its K rows and V rows) per tile; the block ids come from the
// block table through scalar loads, one tile ahead of the load they steer.
constexpr int kMaxTableBlocks = 1 << 24;  // block-table width accepted (keeps token positions in int)
// Largest per-lane sum of a tile's exponentials accepted without taking the
// tile's column max (each exponential is then at most this, 2^8).
constexpr float kSumLimit = 256.f;
constexpr int kQueueWords = 16;      // workspace: 8 queue counters, finished workgroups, drained queues
constexpr int kDoneWord = 8;
constexpr int kDrainedWord = 9;

// s_waitcnt vmcnt(n) with the other counters left free (n < 16).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 16, "vmcnt immediate");
  __builtin_amdgcn_s_waitcnt(0x0F70 | N);
}

// s_waitcnt lgkmcnt(0) with the other counters left free.
__device__ __forceinline__ void wait_lgkmcnt0() { __builtin_amdgcn_s_waitcnt(0xC07F); }

// Workgroup barrier without the memory fence of __syncthreads: the caller
// has already waited for exactly the loads it needs.  The empty asm keeps the
// compiler from moving memory accesses across it.
__device__ __forceinline__ void bare_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Index of the XCD (accelerator complex die) running this wave: hardware
// register XCC_ID (id 20), bits 0-3.
__device__ __forceinline__ unsigned xcd_id() {
  return static_cast<unsigned>(__builtin_amdgcn_s_getreg((31 << 11) | 20)) & 7u;
}

// What one launch of the attention kernel computes.
//   kFull:   each request's queries over all of its keys (causal).
//   kShared: first half of a split over a prefix of kv_split keys that every
//            request shares (same blocks, all before any query): every query
//            row of the batch over keys [0, kv_split) of request 0's table, no
//            mask; the unnormalised O, the running max and the sum go to
//            part_o / part_ml instead of out.
//   kSuffix: second half: each request's queries over keys [kv_split, L)
//            (causal), starting from the state kShared left, normalised into out.
// Splitting this way reads the shared K/V once per column tile of the whole
// batch instead of once per request (the log-sum-exp merge of the two halves
// is exact up to rounding).
//   kFused:  the same split in one launch: every item is 256 columns of the
//            whole batch's packed query rows (like kShared); it runs the
//            kv_split / 64 tiles every request shares, then, for each
//            request its rows belong to, that request's own tiles from
//            kv_split on, masked to that request's columns.  No partial
//            state leaves the workgroup.
enum AttnMode { kFull = 0, kShared = 1, kSuffix = 2, kFused = 3 };

// kFused: per item, the request tiles after the shared ones, in LDS.
constexpr int kFusedTiles = 2048;

template <int D, int MODE>
__global__ __launch_bounds__(kThreads, 1) void paged_attn_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_pool,
    const uint16_t* __restrict__ v_pool, int num_blocks, const int32_t* __restrict__ block_tables,
    int max_blocks, const int32_t* __restrict__ cu_q, const int32_t* __restrict__ seq_lens, int n_req,
    int Hq, int Hkv, int n_col_tiles, unsigned n_items, float scale_log2, uint16_t* __restrict__ out,
    unsigned* __restrict__ queue, int kv_split, float* __restrict__ part_o, float* __restrict__ part_ml,
    int part_rows) {
  constexpr int kDch = D / 16;                    // 16-wide contraction chunks of Q.K^T
  constexpr int kDt = D / 32;                     // 32-row output tiles of O^T
  constexpr int kRowBytes = D * 2;                // one K row in LDS
  constexpr int kKch = D / 8;                     // 16-byte chunks per K row
  constexpr int kKTileBytes = kKeys * kRowBytes;  // one K tile
  constexpr int kVBlockBytes = D * 32;            // one [D][16] V block
  constexpr int kVTileBytes = kTileBlocks * kVBlockBytes;
  constexpr int kStageBytes = kKTileBytes + kVTileBytes;
  constexpr int kSlabBytes = kBlock * D * 2;      // one (block, kv head) slab in a pool
  constexpr int kKInsts = kKTileBytes / 1024 / kWaves;  // 1 KB direct loads per wave per tile
  constexpr int kVInsts = kVTileBytes / 1024 / kWaves;
  constexpr int kLoads = kKInsts + kVInsts;
  static_assert(kKInsts >= 1 && kVInsts >= 1 && kWaves == 2 * kTileBlocks, "load split");
  static_assert(kStages == 4, "ring: two tiles in flight plus two being read");
  __shared__ __attribute__((aligned(16))) uint8_t ring[kStages * kStageBytes];
  __shared__ int s_item[2];
  // kFused: tile T_s + i of an item is tile f_tt[i] of request r_a + f_rel[i],
  // whose keys at or past f_lim[i] no row of the item sees.
  constexpr int kFT = MODE == kFused ? kFusedTiles : 1;
  __shared__ int f_rel[kFT], f_tt[kFT], f_lim[kFT];
  __shared__ int f_count;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int n = lane & 31, hh = lane >> 5;
  const int G = Hq / Hkv;
  const size_t slab_stride = size_t(Hkv) * kSlabBytes;

  // Item queues.  Queue x holds items [x*per + min(x, extra), ...) of
  // per + (x < extra) items; fetch() (lane 0 of wave 0 only) returns the next
  // item, or -1 once every queue is drained.  The workgroup that takes the
  // last item of a queue counts it in queue[kDrainedWord]; once the home queue
  // is drained, that count (one round trip) tells whether any queue still
  // holds items.  Without it, the walk over the drained queues (one contended
  // atomic each, about 2 us) sat in front of every workgroup's last item.
  const unsigned home = xcd_id(), per = n_items >> 3, extra = n_items & 7u;
  const unsigned nonempty = per > 0 ? 8u : extra;  // queues holding at least one item
  // With no more items than workgroups (grid = items), workgroup b takes
  // item b/8 of queue b%8 (the queue of the XCD it is dispatched to in
  // round-robin order) and nothing else: no queue atomics, no exit count,
  // and the workspace is left untouched.  Queue x has exactly as many items
  // as there are such workgroups.
  unsigned qsel = 0;  // next queue to try, home first (9: the one-item-each mode)
  auto fetch = [&]() -> int {
    while (qsel < 8u) {
      const unsigned x = (home + qsel) & 7u;
      const unsigned size = per + (x < extra ? 1u : 0u), base = x * per + min(x, extra);
      const unsigned i = __hip_atomic_fetch_add(queue + x, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (i + 1 == size) __hip_atomic_fetch_add(queue + kDrainedWord, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (i < size) return int(base + i);
      ++qsel;
      if (qsel == 1u &&
          __hip_atomic_load(queue + kDrainedWord, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= nonempty)
        qsel = 8u;
    }
    return -1;
  };

  // This wave's direct loads of a tile: all from pool block wave/2 of the tile.
  // LDS slot (row m, slot p) of a K tile holds chunk k_slot(m, p) of key
  // key_row(m); slot (d, p) of a V block holds half v_slot(d, p) of row d.
  uint32_t koff[kKInsts], voff[kVInsts];
#pragma unroll
  for (int i = 0; i < kKInsts; ++i) {
    const int g = wave * kKInsts + i;
    const int m = g * (1024 / kRowBytes) + lane / kKch;
    koff[i] = uint32_t((key_row(m) & 15) * kRowBytes + k_slot<D>(m, lane % kKch) * 16);
  }
#pragma unroll
  for (int i = 0; i < kVInsts; ++i) {
    const int g = wave * kVInsts + i;
    const int d = (g * 1024 % kVBlockBytes) / 32 + (lane >> 1);
    voff[i] = uint32_t(d * 32 + v_slot(d, lane & 1) * 16);
  }
  const int my_blk = wave >> 1;
  const bool lag = wave >= kWaves / 2;

  if (tid == 0) {
    if (n_items <= gridDim.x) {
      const unsigned x = blockIdx.x & 7u;
      s_item[0] = int(x * per + min(x, extra) + (blockIdx.x >> 3));
      qsel = 9u;  // later fetches return -1
    } else {
      s_item[0] = fetch();
    }
    wait_lgkmcnt0();
  }
  __syncthreads();

  // Ring stages are numbered by a tile count running across items, so the
  // first tiles of an item never land in the stage the previous item still
  // reads.
  int tbase = 0;
  for (int it = 0;; ++it) {
    const int w = __builtin_amdgcn_readfirstlane(s_item[it & 1]);
    if (w < 0) break;
    // kFused numbers items kv-head-major (the items of one kv head share the
    // prefix blocks, under one XCD's L2).
    const int tile = MODE == kFused ? int(unsigned(w) % unsigned(n_col_tiles))
                                    : n_col_tiles - 1 - int(unsigned(w) % unsigned(n_col_tiles));
    const unsigned rest = unsigned(w) / unsigned(n_col_tiles);
    const int kvh = MODE == kFused ? int(rest) : int(rest % unsigned(Hkv));
    const int r = MODE == kShared || MODE == kFused ? 0 : int(rest / unsigned(Hkv));
    // First key tile of this launch (the suffix half starts at kv_split).
    const int t0 = MODE == kSuffix ? kv_split / kKeys : 0;
    // This item's lengths and the block ids of its first three tiles are
    // loaded together: one round trip for all.  A block id is loaded
    // unconditionally (clamped into the table row) and checked where it is
    // used, so that no wait follows the scalar load.
    const int32_t* bt = block_tables + size_t(r) * max_blocks;
    auto raw_id = [&](int tl) { return bt[min((t0 + tl) * kTileBlocks + my_blk, max_blocks - 1)]; };
    // kFused: request (relative to r_a) and tile of item tile tl.
    auto fused_src = [&](int tl, int& rel, int& tt) {
      if (tl < kv_split / kKeys) {
        rel = 0;
        tt = tl;
      } else {
        rel = __builtin_amdgcn_readfirstlane(f_rel[tl - kv_split / kKeys]);
        tt = __builtin_amdgcn_readfirstlane(f_tt[tl - kv_split / kKeys]);
      }
    };
    // The shared half treats the whole batch as one request whose queries all
    // follow the kv_split shared keys.
    const int q0 = MODE == kShared || MODE == kFused ? 0 : cu_q[r];
    const int q_end = MODE == kShared || MODE == kFused ? cu_q[n_req] : cu_q[r + 1];
    const int L_in = MODE == kShared || MODE == kFused ? kv_split + (q_end - q0) : seq_lens[r];
    const int raw_id0 = raw_id(0), raw_id1 = raw_id(1);
    int raw_next = raw_id(2);  // raw id of the next tile to issue after tile 1
    // First use of all six values at once: the loads are issued together and
    // waited for once.
    asm volatile("" : : "s"(q0), "s"(q_end), "s"(L_in), "s"(raw_id0), "s"(raw_id1), "s"(raw_next));
    // In the split modes, rows past the partial-state buffer are not computed.
    const int q_len = MODE == kFull || MODE == kFused ? q_end - q0 : min(q_end, part_rows) - q0;
    const int n_cols = q_len * G;
    const int col0 = tile * kCols;
    const int L = MODE == kShared || MODE == kFused ? L_in : min(L_in, max_blocks * kBlock);
    if (q_len <= 0 || col0 >= n_cols || q_len > L) {  // nothing to do for this item
      if (tid == 0) {
        s_item[(it + 1) & 1] = fetch();
        wait_lgkmcnt0();
      }
      __syncthreads();
      continue;
    }
    const int qstart = L - q_len;  // position of the request's first query

    const int T_s = kv_split / kKeys;  // kFused: tiles every request shares (at least 3)
    int r_a = 0, my_rel = 0, my_pos = 0;
    // This lane's query column (padding columns repeat the last valid one).
    const int col = col0 + wave * kColsPerWave + n;
    const bool col_valid = col < n_cols;
    const int colc = col_valid ? col : n_cols - 1;
    const int t = colc / G;
    const int pos = qstart + t;
    const size_t qrow = (size_t(q0 + t) * Hq + size_t(kvh) * G + (colc - t * G)) * D;

    const int wave_first = col0 + wave * kColsPerWave;
    const bool wave_active = wave_first < n_cols;
    const int wave_pos_min = qstart + min(wave_first, n_cols - 1) / G;
    const int wg_pos_max = qstart + min(col0 + kCols - 1, n_cols - 1) / G;
    // Keys at or past key_lim are masked everywhere (and their V rows zeroed).
    const int key_lim = MODE == kShared ? kv_split : wg_pos_max + 1;
    // Tiles of this launch (kFused: the shared ones until the item's list is
    // read after the first barrier).
    int n_tiles = MODE == kFused ? T_s : (key_lim - 1) / kKeys + 1 - t0;
    const int n_blk_used = (key_lim + kBlock - 1) / kBlock;  // <= ceil(L / 16) <= max_blocks
    // Last tile (counted from t0) holding a key some column of this wave sees
    // (-1: no column).
    int wave_last =
        !wave_active ? -1
        : MODE == kShared || MODE == kFused ? n_tiles - 1
                          : (qstart + min(wave_first + kColsPerWave - 1, n_cols - 1) / G) / kKeys - t0;

    bf16x8 qf[kDch];
#pragma unroll
    for (int kc = 0; kc < kDch; ++kc) qf[kc] = as_bf16x8(*(const u32x4*)(q + qrow + kc * 16 + hh * 8));
    // kFused: block id of this wave in item tile tl (shared tiles from any
    // request's table, request tiles from the owner's).
    auto fused_raw = [&](int tl) {
      int rel, tt;
      fused_src(tl, rel, tt);
      return block_tables[size_t(r_a + rel) * max_blocks + min(tt * kTileBlocks + my_blk, max_blocks - 1)];
    };


    const uint8_t* kbase = reinterpret_cast<const uint8_t*>(k_pool) + size_t(kvh) * kSlabBytes;
    const uint8_t* vbase = reinterpret_cast<const uint8_t*>(v_pool) + size_t(kvh) * kSlabBytes;
    // Pool block of this wave in tile tl, from the raw table entry; unusable
    // ids read block 0 instead (stray K rows only meet masked scores, stray V
    // rows past key_lim are zeroed below).
    auto usable = [&](int tl, int id) {
      if constexpr (MODE == kFused) return (id >= 0 && id < num_blocks) ? id : 0;
      return ((t0 + tl) * kTileBlocks + my_blk < n_blk_used && id >= 0 && id < num_blocks) ? id : 0;
    };
    auto stage = [&](int tl) { return ring + (unsigned(tbase + tl) % unsigned(kStages)) * kStageBytes; };
    auto issue_tile = [&](int tl, int raw) {
      const int id = usable(tl, raw);
      uint8_t* st = stage(tl);
      const uint8_t* ksrc = kbase + size_t(id) * slab_stride;
      const uint8_t* vsrc = vbase + size_t(id) * slab_stride;
#pragma unroll
      for (int i = 0; i < kKInsts; ++i) global_to_lds16(ksrc + koff[i], st + (wave * kKInsts + i) * 1024);
#pragma unroll
      for (int i = 0; i < kVInsts; ++i)
        global_to_lds16(vsrc + voff[i], st + kKTileBytes + (wave * kVInsts + i) * 1024);
    };
    // Zero the V rows of keys >= key_lim in a V tile (only the tile crossing it).
    auto zero_v_tail = [&](int j0, uint8_t* sV, int key_lim) {
      for (int slot = tid; slot < kVTileBytes / 16; slot += kThreads) {
        const int kb = slot / (2 * D), d = (slot % (2 * D)) >> 1, p = slot & 1;
        const int nvalid = key_lim - (j0 + kb * kBlock + v_slot(d, p) * 8);
        if (nvalid < 8) {
          u32x4* ptr = (u32x4*)(sV + kb * kVBlockBytes + d * 32 + p * 16);
          u32x4 v = *ptr;
#pragma unroll
          for (int e = 0; e < 4; ++e)
            v[e] &= (2 * e < nvalid ? 0x0000FFFFu : 0u) | (2 * e + 1 < nvalid ? 0xFFFF0000u : 0u);
          *ptr = v;
        }
      }
    };

    f32x16 o[kDt];
#pragma unroll
    for (int dt = 0; dt < kDt; ++dt)
#pragma unroll
      for (int i = 0; i < 16; ++i) o[dt][i] = 0.f;
    float m_used = -INFINITY;  // max (log2 units) the exponentials of this column are taken against
    float l_run = 0.f;         // this lane half's share of the column's exponential sum
    const size_t prow = qrow / D;  // (query row, q head) of this lane's column
    if constexpr (MODE == kSuffix) {
      // Continue from the shared half's state (loaded with Q, waited for with
      // the first tiles).  Lane half 0 carries the whole sum.
      m_used = part_ml[prow * 2];
      l_run = hh == 0 ? part_ml[prow * 2 + 1] : 0.f;
#pragma unroll
      for (int dt = 0; dt < kDt; ++dt)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const f32x4 v = *(const f32x4*)(part_o + prow * D + dt * 32 + g4 * 8 + hh * 4);
#pragma unroll
          for (int e = 0; e < 4; ++e) o[dt][g4 * 4 + e] = v[e];
        }
    }
    bf16x8 pb[kTileBlocks];    // P of the tile whose V^T P^T is still due
    f32x16 sc0, sc1;           // scores of the tile whose softmax is next

    // Softmax step of the score tile starting at key j0: causal mask, then
    // P = exp2(S * scale_log2 - m_used), rounded to bf16 for the V^T P^T
    // product while the row sum adds the fp32 values.  m_used is the column
    // max the exponentials were last rescaled to.  The step is accepted as
    // long as every lane's sum of its exponentials lies in [0, 2^8] (so no
    // single one exceeds 2^8, the headroom the fp32 accumulators are given);
    // otherwise -- on the first tile (`first`: m_used is still -inf), or when
    // the max has grown -- the tile's column max is taken, O and the sum are
    // rescaled to it and the exponentials recomputed.
    // Lane half hh holds keys j0 + (e>>3)*16 + 8*hh + (e&7) [+32] of the tile.
    auto softmax = [&](int j0, bool first, int fused_thr) __attribute__((always_inline)) {
      if (MODE == kFused && fused_thr != INT_MAX) {  // a request tile: its own rows, causal
        const int rel = fused_thr;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int k = (e >> 3) * 16 + (e & 7);
          sc0[e] = k > rel ? -INFINITY : sc0[e];
          sc1[e] = k + 32 > rel ? -INFINITY : sc1[e];
        }
      }
      if (MODE != kShared && MODE != kFused && j0 + kKeys - 1 > wave_pos_min) {  // causal
        const int rel = pos - j0 - hh * 8;  // key (e>>3)*16 + (e&7) [+32] is visible iff <= rel
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int k = (e >> 3) * 16 + (e & 7);
          sc0[e] = k > rel ? -INFINITY : sc0[e];
          sc1[e] = k + 32 > rel ? -INFINITY : sc1[e];
        }
      }
      if (MODE == kShared && j0 + kKeys > key_lim) {  // keys past the shared prefix
        int lim = key_lim - j0 - hh * 8;
        asm volatile("" : "+v"(lim));  // computed here: hoisted, the 32 compares would pin 64 SGPRs
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int k = (e >> 3) * 16 + (e & 7);
          sc0[e] = k >= lim ? -INFINITY : sc0[e];
          sc1[e] = k + 32 >= lim ? -INFINITY : sc1[e];
        }
      }
      if (MODE == kSuffix && j0 < kv_split) {  // keys of the shared prefix: done before
        int lo = kv_split - j0 - hh * 8;
        asm volatile("" : "+v"(lo));  // as above
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int k = (e >> 3) * 16 + (e & 7);
          sc0[e] = k < lo ? -INFINITY : sc0[e];
          sc1[e] = k + 32 < lo ? -INFINITY : sc1[e];
        }
      }
      // Exponentials against the running max m_used, summed per lane half.
      auto exps = [&](float* ls) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sc0[e], scale_log2, -m_used));
          const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sc1[e], scale_log2, -m_used));
          pb[e >> 3][e & 7] = (__bf16)p0;
          pb[2 + (e >> 3)][e & 7] = (__bf16)p1;
          ls[e & 3] = e < 4 ? p0 + p1 : ls[e & 3] + (p0 + p1);
        }
        // The bf16 operands are formed here, not after the acceptance test:
        // sunk past it, all 32 fp32 exponentials would stay live across it.
        asm volatile("" : "+v"(pb[0]), "+v"(pb[1]), "+v"(pb[2]), "+v"(pb[3]));
      };
      float ls[4];
      float tsum = 0.f;
      bool slow = first;
      if (!first) {
        exps(ls);
        tsum = (ls[0] + ls[1]) + (ls[2] + ls[3]);
        // Accepted unless some lane's sum exceeds kSumLimit or is not a
        // number (an overflow, or -inf - -inf).
        slow = __ballot(!(tsum <= kSumLimit)) != 0;
      }
      if (slow) {
        float mx, mx2;
        asm("v_max3_f32 %0, %1, %2, %3\n\t"
            "v_max3_f32 %0, %0, %4, %5\n\t"
            "v_max3_f32 %0, %0, %6, %7\n\t"
            "v_max3_f32 %0, %0, %8, %9\n\t"
            "v_max3_f32 %0, %0, %10, %11\n\t"
            "v_max3_f32 %0, %0, %12, %13\n\t"
            "v_max3_f32 %0, %0, %14, %15\n\t"
            "v_max3_f32 %0, %0, %16, %17"
            : "=&v"(mx)
            : "v"(sc0[0]), "v"(sc1[0]), "v"(sc0[1]), "v"(sc1[1]), "v"(sc0[2]), "v"(sc1[2]), "v"(sc0[3]),
              "v"(sc1[3]), "v"(sc0[4]), "v"(sc1[4]), "v"(sc0[5]), "v"(sc1[5]), "v"(sc0[6]), "v"(sc1[6]),
              "v"(sc0[7]), "v"(sc1[7]), "v"(sc0[8]));
        asm("v_max3_f32 %0, %1, %2, %3\n\t"
            "v_max3_f32 %0, %0, %4, %5\n\t"
            "v_max3_f32 %0, %0, %6, %7\n\t"
            "v_max3_f32 %0, %0, %8, %9\n\t"
            "v_max3_f32 %0, %0, %10, %11\n\t"
            "v_max3_f32 %0, %0, %12, %13\n\t"
            "v_max3_f32 %0, %0, %14, %15\n\t"
            "v_max3_f32 %0, %0, %16, %0"
            : "=&v"(mx2)
            : "v"(mx), "v"(sc1[8]), "v"(sc0[9]), "v"(sc1[9]), "v"(sc0[10]), "v"(sc1[10]), "v"(sc0[11]),
              "v"(sc1[11]), "v"(sc0[12]), "v"(sc1[12]), "v"(sc0[13]), "v"(sc1[13]), "v"(sc0[14]),
              "v"(sc1[14]), "v"(sc0[15]), "v"(sc1[15]));
        mx = mx2;
        mx = max_across_halves(mx) * scale_log2;
        const float m_new = fmaxf(m_used, mx);
        const float alpha = __builtin_amdgcn_exp2f(m_used - m_new);
        m_used = m_new;
        l_run *= alpha;
#pragma unroll
        for (int dt = 0; dt < kDt; ++dt)
#pragma unroll
          for (int e = 0; e < 16; ++e) o[dt][e] *= alpha;
        exps(ls);
        tsum = (ls[0] + ls[1]) + (ls[2] + ls[3]);
      }
      l_run += tsum;
    };

    // One matrix-core phase: O += V(sV) P over the tile's pool blocks
    // (kTileBlocks * kDt products), then S = K(sK) Q^T (2 * kDch products),
    // as one software-pipelined stream whose LDS operands are read kPrefetch
    // products ahead, so that a lone wave keeps the matrix core busy.
    constexpr int kPvSteps = kTileBlocks * kDt, kQkSteps = 2 * kDch, kPrefetch = 4;
    auto m_phase = [&](auto with_pv, auto with_qk, const uint8_t* sV, const uint8_t* sK) {
      constexpr int first = decltype(with_pv)::value ? 0 : kPvSteps;
      constexpr int last = decltype(with_qk)::value ? kPvSteps + kQkSteps : kPvSteps;
      auto operand = [&](int st) -> bf16x8 {
        if (st < kPvSteps) {
          const int b = st / kDt, d = (st % kDt) * 32 + n;
          return *(const bf16x8*)(sV + b * kVBlockBytes + d * 32 + (v_slot(d, hh) << 4));
        }
        const int u = st - kPvSteps, m = (u & 1) * 32 + n;
        return *(const bf16x8*)(sK + m * kRowBytes + (k_slot<D>(m, (u >> 1) * 2 + hh) << 4));
      };
      // Raised issue priority for the phase: when the partner wave's softmax
      // and this wave's next product are both ready, the product goes first,
      // so the matrix core does not wait behind a run of vector instructions
      // (1-2.5% faster than equal priority on llama8b, qwen7b, large and
      // sweep100).  The scheduling barriers keep the phase's instructions
      // between the two priority changes.
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_setprio(1);
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (decltype(with_qk)::value) {
#pragma unroll
        for (int e = 0; e < 16; ++e) { sc0[e] = 0.f; sc1[e] = 0.f; }
      }
      bf16x8 buf[kPrefetch];
#pragma unroll
      for (int st = first; st < first + kPrefetch && st < last; ++st) buf[st % kPrefetch] = operand(st);
#pragma unroll
      for (int st = first; st < last; ++st) {
        const bf16x8 a = buf[st % kPrefetch];
        if (st + kPrefetch < last) buf[st % kPrefetch] = operand(st + kPrefetch);
        if (st < kPvSteps) {
          const int dt = st % kDt;
          o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[st / kDt], o[dt], 0, 0, 0);
        } else {
          const int u = st - kPvSteps;
          if (u & 1) sc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[u >> 1], sc1, 0, 0, 0);
          else sc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[u >> 1], sc0, 0, 0, 0);
        }
      }
      // Pin the pipelined order for the scheduler (mask 0x100: LDS reads,
      // 0x008: matrix-core ops): kPrefetch reads, then one product per read,
      // then the last kPrefetch products.
      constexpr int steps = last - first, lead = steps < kPrefetch ? steps : kPrefetch;
      __builtin_amdgcn_sched_group_barrier(0x100, lead, 0);
#pragma unroll
      for (int st = 0; st < steps - lead; ++st) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, lead, 0);
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_setprio(0);
      __builtin_amdgcn_sched_barrier(0);
    };
    using yes = std::true_type;
    using no = std::false_type;

    // Ping-pong schedule.  Every wave runs the same phase sequence
    //   M_0 = [S(0) = K(0) Q^T]
    //   V_0 = [softmax S(0) -> P(0)]
    //   M_j = [O += V(j-1) P(j-1); S(j) = K(j) Q^T]   j = 1 .. n_tiles-1
    //   V_j = [softmax S(j) -> P(j)]
    //   M_n = [O += V(n-1) P(n-1)]
    // with a workgroup barrier before every phase.  Waves kWaves/2 .. kWaves-1
    // pass one extra barrier first (and waves 0 .. kWaves/2-1 one at the
    // end), so the second half runs one phase behind the first: while one
    // wave of a SIMD issues matrix-core work (M) its partner runs the vector
    // softmax (V).
    //
    // Counting this item's barriers, the first half runs phase number p (M_j
    // is p = 2j, V_j is p = 2j+1) after barrier p and the second half after
    // barrier p+1.  Hence:
    //   - every wave waits for its own loads of tile j before the barrier
    //     that opens V_{j-1}: barrier 2j-1 or 2j, so all of tile j is in LDS
    //     by barrier 2j, where the first half starts M_j;
    //   - the V tail of tile j is zeroed at the start of M_j (after barrier
    //     2j or 2j+1, once tile j is complete) and read in M_{j+1} (after
    //     barrier 2j+2 or 2j+3);
    //   - tile j+2 is issued at the start of V_j (after barrier 2j+1 or
    //     2j+2), into the stage of tile j-2, whose last reader M_{j-1} ended
    //     by barrier 2j everywhere.
    // The ring thus holds tiles j-1 (V still due), j and j+1 (in flight
    // since V_{j-1}) during M_j, and j+2 from V_j on.  The loads are issued
    // in the softmax phase rather than at the start of M_j so that their
    // issue stays off the matrix-core phase, which sets the pace: 2-7%
    // faster on llama8b, qwen7b, large and the hit-rate sweep than issuing
    // at M_j, with a tile of lead still enough that the waits stay short.
    // Across items the stage count runs on: when the first half starts the
    // next item, the second half may still be in M_n of this one, which
    // reads the stage of tile n-1, while the next item's tiles 0, 1 and 2 go
    // to the stages after it.
    auto wait_tile = [&](int) { wait_vmcnt<0>(); };  // the newest loads of this wave are the tile's
    auto begin_m = [&](int j) {
      bare_barrier();
      if (MODE == kFused && j == 0) {  // the item's list is complete (wave 0 waited before this barrier)
        n_tiles = T_s + __builtin_amdgcn_readfirstlane(f_count);
        wave_last = wave_active ? n_tiles - 1 : -1;
      }
      if (MODE == kFused && j >= T_s && j < n_tiles) {
        const int i = j - T_s;
        const int tt = __builtin_amdgcn_readfirstlane(f_tt[i]), lim = __builtin_amdgcn_readfirstlane(f_lim[i]);
        if (tt * kKeys + kKeys > lim) {
          zero_v_tail(tt * kKeys, stage(j) + kKTileBytes, lim);
          wait_lgkmcnt0();
        }
      } else if (MODE != kFused && j < n_tiles && (t0 + j) * kKeys + kKeys > key_lim) {
        zero_v_tail((t0 + j) * kKeys, stage(j) + kKTileBytes, key_lim);
        wait_lgkmcnt0();  // zeros in LDS before the next barrier
      }
    };
    // The block id of tile j+3 (issued in V_{j+1}) is loaded at the start of
    // V_j, right after tile j+2 is issued with the previous one: no LDS read
    // follows until the next phase, so the scalar load (which shares lgkmcnt
    // with LDS reads) has landed before anything waits on lgkmcnt.
    auto prefetch_id = [&](int j) {
      if (j + 3 < n_tiles) raw_next = MODE == kFused ? fused_raw(j + 3) : raw_id(j + 3);
    };

    issue_tile(0, raw_id0);
    if (1 < n_tiles) issue_tile(1, raw_id1);
    // kFused: with the first tiles and Q in flight, find the requests of the
    // item's rows, this lane's request and position, and (wave 0) the list of
    // request tiles; tiles 0-2 are shared, so request 0's table gave their ids.
    // Scalar loads only: they do not queue behind the tiles' vector loads.
    if constexpr (MODE == kFused) {
      const int row_a = col0 / G, row_b = min(col0 + kCols - 1, n_cols - 1) / G;
      // r_a: the largest request whose first row is at or before row_a
      int lo = 0, hi = n_req;  // cu_q[lo] <= row_a < cu_q[hi]
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (cu_q[mid] <= row_a) lo = mid;
        else hi = mid;
      }
      r_a = lo;
      const int col_l = min(col0 + wave * kColsPerWave + n, n_cols - 1);
      const int row_l = col_l / G;
      int n_list = 0;
      // requests r_a, r_a + 1, ... while their rows start at or before row_b
      for (int rr = r_a; rr < n_req; ++rr) {
        const int b0 = cu_q[rr];
        if (b0 > row_b) break;
        const int b1 = cu_q[rr + 1];
        const int lo_row = max(b0, row_a), hi_row = min(b1 - 1, row_b);
        if (lo_row > hi_row) continue;  // no row of this item (or an empty request)
        const int Lr = min(seq_lens[rr], max_blocks * kBlock);
        if (row_l >= b0 && row_l < b1) {
          my_rel = rr - r_a;
          my_pos = Lr - (b1 - b0) + (row_l - b0);
        }
        // keys the item's rows of rr see end at lim; its tiles T_s .. go to the list
        const int lim = Lr - (b1 - b0) + (hi_row - b0) + 1;
        const int cnt = min(max(0, (lim + kKeys - 1) / kKeys - T_s), kFusedTiles - n_list);
        if (wave == 0) {
          for (int k = lane; k < cnt; k += 64) {
            f_rel[n_list + k] = rr - r_a;
            f_tt[n_list + k] = T_s + k;
            f_lim[n_list + k] = lim;
          }
        }
        n_list += cnt;
      }
      if (wave == 0) {
        if (lane == 0) f_count = n_list;
        wait_lgkmcnt0();  // the list is in LDS before the barrier that opens M_0
      }
    }
    if (tid == 0) {  // the next item, fetched while the first tiles load
      s_item[(it + 1) & 1] = fetch();
      wait_lgkmcnt0();
    }
    // Q and tiles 0 and 1 in (before the second half's extra barrier, which
    // stands in for the barrier opening V_{-1}).
    wait_vmcnt<0>();
    if (lag) bare_barrier();
    // kFused: mask threshold of item tile j for this lane (INT_MAX: a shared
    // tile, all keys visible) and the tile's first key in its request.
    auto fused_thr = [&](int j, int& j0) {
      if (j < T_s) {
        j0 = j * kKeys;
        return INT_MAX;
      }
      const int rel = __builtin_amdgcn_readfirstlane(f_rel[j - T_s]);
      j0 = __builtin_amdgcn_readfirstlane(f_tt[j - T_s]) * kKeys;
      return rel == my_rel ? my_pos - j0 - hh * 8 : -1;
    };
    auto soft = [&](int j, bool first) __attribute__((always_inline)) {
      if constexpr (MODE == kFused) {
        int j0;
        const int th = fused_thr(j, j0);
        softmax(j0, first, th);
      } else {
        softmax((t0 + j) * kKeys, first, INT_MAX);
      }
    };
    begin_m(0);
    if (0 <= wave_last) m_phase(no(), yes(), stage(0), stage(0));
    if (n_tiles > 1) wait_tile(1);
    bare_barrier();
    if (2 < n_tiles) issue_tile(2, raw_next);
    prefetch_id(0);
    if (0 <= wave_last) soft(0, MODE != kSuffix);
    for (int j = 1; j < n_tiles; ++j) {
      begin_m(j);
      // Tiles past the wave's last visible key are skipped; the step right
      // after it still adds P(j-1) (its S(j) product is wasted and ignored).
      if (j - 1 <= wave_last) m_phase(yes(), yes(), stage(j - 1) + kKTileBytes, stage(j));
      if (j + 1 < n_tiles) wait_tile(j + 1);
      bare_barrier();
      if (j + 2 < n_tiles) issue_tile(j + 2, raw_next);
      prefetch_id(j);
      if (j <= wave_last) soft(j, false);
    }
    begin_m(n_tiles);
    if (n_tiles - 1 <= wave_last) m_phase(yes(), no(), stage(n_tiles - 1) + kKTileBytes, stage(0));
    if (!lag) bare_barrier();
    tbase += n_tiles;

    if (wave_active) {
      const float l_tot = l_run + __shfl_xor(l_run, 32);
      if constexpr (MODE == kShared) {  // unnormalised O, max and sum for the suffix half
        if (col_valid) {
          if (hh == 0) {
            part_ml[prow * 2] = m_used;
            part_ml[prow * 2 + 1] = l_tot;
          }
#pragma unroll
          for (int dt = 0; dt < kDt; ++dt)
#pragma unroll
            for (int g4 = 0; g4 < 4; ++g4) {
              const f32x4 v = {o[dt][g4 * 4], o[dt][g4 * 4 + 1], o[dt][g4 * 4 + 2], o[dt][g4 * 4 + 3]};
              *(f32x4*)(part_o + prow * D + dt * 32 + g4 * 8 + hh * 4) = v;
            }
        }
      } else if constexpr (D == 128) {
        // The normalised O leaves through LDS.  In the matrix-core layout a
        // lane holds 8-byte pieces of one output row, so direct stores put 16
        // bytes of 32 different rows into every instruction; those scattered
        // stores held up the item boundary (timed without them, llama8b and
        // large ran 16% and 8% faster).  Each wave writes its 32 rows, 64
        // dimensions at a time, into its 4 KiB of the ring stage the next
        // item's tile 2 will take, then stores whole 128-byte half rows, 8
        // lanes per half row.  That stage (tile n-2's) is free: its last
        // reader M_{n-1} ended by barrier 2n everywhere, and the next item
        // writes it only in its V_0, after both halves have passed here.
        // 16-byte chunks are XOR-swizzled by row against bank conflicts.
        const float inv = 1.f / l_tot;
        uint8_t* tb = stage(2) + wave * (kStageBytes / kWaves);
        static_assert(kStageBytes / kWaves >= kColsPerWave * 128, "transpose area");
        size_t orow4[4];  // output row of the 4 rows this lane stores
        bool ok4[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int c = col0 + wave * kColsPerWave + r * 8 + (lane >> 3);
          ok4[r] = c < n_cols;
          const int tr = c / G;
          orow4[r] = (size_t(q0 + tr) * Hq + size_t(kvh) * G + (c - tr * G)) * D;
        }
        const int ch_r = lane & 7;
#pragma unroll
        for (int p = 0; p < kDt / 2; ++p) {
#pragma unroll
          for (int dl = 0; dl < 2; ++dl)
#pragma unroll
            for (int g4 = 0; g4 < 4; ++g4) {
              bf16x4 v;
#pragma unroll
              for (int e = 0; e < 4; ++e) v[e] = (__bf16)(o[2 * p + dl][g4 * 4 + e] * inv);
              const int ch = dl * 4 + g4;
              *(bf16x4*)(tb + n * 128 + ((ch ^ (n & 7)) << 4) + hh * 8) = v;
            }
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int row = r * 8 + (lane >> 3);
            const u32x4 val = *(const u32x4*)(tb + row * 128 + ((ch_r ^ (row & 7)) << 4));
            if (ok4[r]) *(u32x4*)(out + orow4[r] + p * 64 + ch_r * 8) = val;
          }
        }
      } else {
        const float inv = 1.f / l_tot;
        if (col_valid) {
          uint16_t* orow = out + qrow;
#pragma unroll
          for (int dt = 0; dt < kDt; ++dt)
#pragma unroll
            for (int g4 = 0; g4 < 4; ++g4) {
              bf16x4 v;
#pragma unroll
              for (int e = 0; e < 4; ++e) v[e] = (__bf16)(o[dt][g4 * 4 + e] * inv);
              *(bf16x4*)(orow + dt * 32 + g4 * 8 + hh * 4) = v;
            }
        }
      }
    }
  }

  // Every queue is drained.  The last workgroup out clears the counters for
  // the next call on this workspace (no workgroup fetches any more by then).
  // The exit count needs no fence.  Wave 0 (which made every queue atomic of
  // this workgroup) first waits until all its memory operations have
  // completed, so once the last workgroup sees the full count no queue atomic
  // of this launch is in flight.  An acquire-release count, with its L2
  // write-back and invalidate at every workgroup's exit, cost 2-5% of the
  // short launches.  The outputs are published by the end of the kernel.
  if (tid == 0 && qsel != 9u) {  // (qsel is 9 only in the one-item-each mode)
    wait_vmcnt<0>();
    const unsigned done =
        __hip_atomic_fetch_add(queue + kDoneWord, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (done == gridDim.x - 1) {
      for (int i = 0; i <= kDrainedWord; ++i)
        __hip_atomic_store(queue + i, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Compute units of the current device (one persistent workgroup each),
// looked up once per device.
int device_cus() {
  static int cached[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 0;
  if (dev < 64 && cached[dev] > 0) return cached[dev];
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  if (dev < 64) cached[dev] = cus;
  return cus;
}

int launch_status(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess)
    return ilpc::set_error(ILPC_EHIP, "%s: launch failed: %s", what, hipGetErrorString(e));
  return ILPC_OK;
}

}  // namespace

extern "C" int ilpc_kv_append(const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_pool,
                              uint16_t* v_pool, int32_t num_blocks, const int32_t* block_tables,
                              int32_t max_blocks, const int32_t* cu_new, const int32_t* start_pos,
                              int32_t B, int32_t max_new, int32_t Hkv, int32_t D,
                              int32_t block_size, void* stream) {
  using ilpc::set_error;
  if (B < 0 || max_new < 0 || num_blocks < 0 || max_blocks < 1 || Hkv < 1)
    return set_error(ILPC_EINVAL, "ilpc_kv_append: negative or zero size");
  if (block_size != kBlock) return set_error(ILPC_EUNSUP, "ilpc_kv_append: block_size must be 16");
  if (D != 64 && D != 128) return set_error(ILPC_EUNSUP, "ilpc_kv_append: head_dim %d unsupported", D);
  if (B == 0 || max_new == 0) return ILPC_OK;
  if (!k_new || !v_new || !k_pool || !v_pool || !block_tables || !cu_new || !start_pos)
    return set_error(ILPC_EINVAL, "ilpc_kv_append: NULL pointer");
  if (!aligned16(k_new) || !aligned16(v_new) || !aligned16(k_pool) || !aligned16(v_pool))
    return set_error(ILPC_EINVAL, "ilpc_kv_append: K/V buffers must be 16-byte aligned");
  if (B > 65535 || Hkv > 65535) return set_error(ILPC_EUNSUP, "ilpc_kv_append: grid too large");
  const int slots = (max_new + kBlock - 2) / kBlock + 1;  // blocks a run of max_new can touch
  const dim3 grid(slots, Hkv, B);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (D == 128)
    hipLaunchKernelGGL(kv_append_kernel<128>, grid, dim3(256), 0, s, k_new, v_new, k_pool, v_pool,
                       num_blocks, block_tables, max_blocks, cu_new, start_pos, max_new, Hkv);
  else
    hipLaunchKernelGGL(kv_append_kernel<64>, grid, dim3(256), 0, s, k_new, v_new, k_pool, v_pool,
                       num_blocks, block_tables, max_blocks, cu_new, start_pos, max_new, Hkv);
  return launch_status("ilpc_kv_append");
}

namespace {

// Key ranges per (request, kv head) pair for the decode kernel.  With fewer
// pairs than SIMDs on the chip: enough ranges for one wave per SIMD, at most
// one per 32-key step of a 16 * max_blocks-token context (max_blocks = 0: no
// such cap) and at most kMaxSplit.  Once the pairs give every SIMD pair a
// wave, splitting pays only on contexts of at least kSplitLongSteps steps:
// on shorter ones the merge launch costs more than the extra waves gain.
constexpr int kSplitLongSteps = 32;

int decode_auto_split(int64_t B, int64_t Hkv, int64_t max_blocks) {
  const int64_t simds = int64_t(device_cus()) * 4;
  const int64_t pairs = B * Hkv;
  if (simds <= 0 || pairs <= 0 || pairs >= simds) return 1;
  int64_t n = std::min<int64_t>((simds + pairs - 1) / pairs, ilpc::kMaxSplit);
  if (max_blocks > 0) {
    const int64_t steps = (max_blocks * kBlock + 31) / 32;
    if (pairs * 2 >= simds && steps < kSplitLongSteps) return 1;
    n = std::min(n, steps);
  }
  return int(n);
}

bool decode_shaped(int64_t max_q_len, int Hq, int Hkv) { return max_q_len * (Hq / Hkv) <= kDecodeCols; }

}  // namespace

extern "C" int ilpc_attn_workspace_bytes(int32_t B, int32_t max_q_len, int32_t Hq, int32_t Hkv,
                                         int32_t D, size_t* bytes) {
  if (!bytes || B < 0 || max_q_len < 0 || Hq < 1 || Hkv < 1 || D < 1)
    return ilpc::set_error(ILPC_EINVAL, "ilpc_attn_workspace_bytes: bad argument");
  *bytes = kQueueWords * sizeof(unsigned);
  // room for the decode kernel's split partials (the largest split any
  // context length can get) on decode-shaped batches with few pairs
  if (B > 0 && max_q_len > 0 && decode_shaped(max_q_len, Hq, Hkv))
    *bytes += ilpc::decode_split_bytes(B, max_q_len, Hq, Hkv, D, decode_auto_split(B, Hkv, 0));
  return ILPC_OK;
}

namespace {

// Cascade workspace: two queue-counter blocks (one per launch), then the
// partial O [rows, Hq, D] and (max, sum) [rows, Hq, 2] in fp32, where
// rows = B * max_q_len; sections start on 256-byte boundaries.
constexpr size_t kCascadeHead = 256;
size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
size_t cascade_part_o_bytes(int64_t rows, int Hq, int D) { return align256(size_t(rows) * Hq * D * 4); }
size_t cascade_bytes(int64_t rows, int Hq, int D) {
  return kCascadeHead + cascade_part_o_bytes(rows, Hq, D) + align256(size_t(rows) * Hq * 2 * 4);
}

// Argument checks shared by both attention entry points.
int check_attn_args(const char* fn, const uint16_t* q, const uint16_t* k_pool, const uint16_t* v_pool,
                    int32_t num_blocks, const int32_t* block_tables, int32_t max_blocks,
                    const int32_t* cu_q, const int32_t* seq_lens, int32_t B, int32_t max_q_len,
                    int32_t Hq, int32_t Hkv, int32_t D, int32_t block_size, float softmax_scale,
                    const uint16_t* out) {
  using ilpc::set_error;
  if (B < 0 || max_q_len < 0 || num_blocks < 1 || max_blocks < 1 || Hq < 1 || Hkv < 1)
    return set_error(ILPC_EINVAL, "%s: negative or zero size", fn);
  if (block_size != kBlock) return set_error(ILPC_EUNSUP, "%s: block_size must be 16", fn);
  if (D != 64 && D != 128) return set_error(ILPC_EUNSUP, "%s: head_dim %d unsupported", fn, D);
  if (Hq % Hkv != 0 || Hq / Hkv > kMaxGroup)
    return set_error(ILPC_EUNSUP, "%s: Hq %d / Hkv %d unsupported", fn, Hq, Hkv);
  if (!std::isfinite(softmax_scale)) return set_error(ILPC_EINVAL, "%s: softmax_scale is not finite", fn);
  if (max_blocks > kMaxTableBlocks)
    return set_error(ILPC_EUNSUP, "%s: max_blocks %d > %d", fn, max_blocks, kMaxTableBlocks);
  if (B == 0 || max_q_len == 0) return ILPC_OK;
  if (!q || !k_pool || !v_pool || !block_tables || !cu_q || !seq_lens || !out)
    return set_error(ILPC_EINVAL, "%s: NULL pointer", fn);
  if (!aligned16(q) || !aligned16(k_pool) || !aligned16(v_pool) || !aligned16(out))
    return set_error(ILPC_EINVAL, "%s: Q/K/V/out must be 16-byte aligned", fn);
  if (int64_t(B) * max_q_len * (Hq / Hkv) / kCols + 1 > (int64_t(1) << 31) / Hkv)
    return set_error(ILPC_EUNSUP, "%s: grid too large", fn);
  return ILPC_OK;
}

// One persistent launch of mode MODE over `items` work items.
template <int MODE>
int launch_attn(const char* fn, const uint16_t* q, const uint16_t* k_pool, const uint16_t* v_pool,
                int32_t num_blocks, const int32_t* block_tables, int32_t max_blocks, const int32_t* cu_q,
                const int32_t* seq_lens, int32_t B, int32_t Hq, int32_t Hkv, int32_t D, int64_t col_tiles,
                float scale_log2, uint16_t* out, unsigned* queue, int kv_split, float* part_o,
                float* part_ml, int part_rows, hipStream_t s) {
  const int64_t items = col_tiles * Hkv * (MODE == kShared || MODE == kFused ? 1 : B);
  if (items == 0) return ILPC_OK;
  const int cus = device_cus();
  if (cus <= 0) return ilpc::set_error(ILPC_EHIP, "%s: cannot query the device", fn);
  const unsigned grid = unsigned(items < cus ? items : cus);
  if (D == 128)
    hipLaunchKernelGGL((paged_attn_kernel<128, MODE>), dim3(grid), dim3(kThreads), 0, s, q, k_pool, v_pool,
                       num_blocks, block_tables, max_blocks, cu_q, seq_lens, B, Hq, Hkv, int(col_tiles),
                       unsigned(items), scale_log2, out, queue, kv_split, part_o, part_ml, part_rows);
  else
    hipLaunchKernelGGL((paged_attn_kernel<64, MODE>), dim3(grid), dim3(kThreads), 0, s, q, k_pool, v_pool,
                       num_blocks, block_tables, max_blocks, cu_q, seq_lens, B, Hq, Hkv, int(col_tiles),
                       unsigned(items), scale_log2, out, queue, kv_split, part_o, part_ml, part_rows);
  return launch_status(fn);
}

}  // namespace

extern "C" int ilpc_paged_prefill_attn(const uint16_t* q, const uint16_t* k_pool,
                                       const uint16_t* v_pool, int32_t num_blocks,
                                       const int32_t* block_tables, int32_t max_blocks,
                                       const int32_t* cu_q, const int32_t* seq_lens, int32_t B,
                                       int32_t max_q_len, int32_t Hq, int32_t Hkv, int32_t D,
                                       int32_t block_size, float softmax_scale, uint16_t* out,
                                       void* workspace, size_t workspace_bytes, void* stream) {
  static const char* fn = "ilpc_paged_prefill_attn";
  int rc = check_attn_args(fn, q, k_pool, v_pool, num_blocks, block_tables, max_blocks, cu_q, seq_lens, B,
                           max_q_len, Hq, Hkv, D, block_size, softmax_scale, out);
  if (rc != ILPC_OK || B == 0 || max_q_len == 0) return rc;
  if (!workspace || workspace_bytes < kQueueWords * sizeof(unsigned) || !aligned16(workspace))
    return ilpc::set_error(ILPC_EINVAL, "%s: workspace must be %zu bytes, 16-byte aligned", fn,
                           kQueueWords * sizeof(unsigned));
  // Decode-shaped batches go to the one-wave-per-pair kernel: split into key
  // ranges when the pairs are fewer than the SIMDs and the workspace has room
  // for the partials (after the queue counters), unsplit when the pairs at
  // least fill the compute units.
  if (decode_shaped(max_q_len, Hq, Hkv)) {
    const float scale_log2 = softmax_scale * 1.4426950408889634f;
    const int n_split = decode_auto_split(B, Hkv, max_blocks);
    const size_t head = kQueueWords * sizeof(unsigned);
    if (n_split > 1 && workspace_bytes >= head + ilpc::decode_split_bytes(B, max_q_len, Hq, Hkv, D, n_split))
      return ilpc::launch_decode_attn(q, k_pool, v_pool, num_blocks, block_tables, max_blocks, cu_q, seq_lens,
                                      B, max_q_len, Hq, Hkv, D, scale_log2, out, n_split,
                                      reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) + head), stream);
    if (int64_t(B) * Hkv >= device_cus())
      return ilpc::launch_decode_attn(q, k_pool, v_pool, num_blocks, block_tables, max_blocks, cu_q, seq_lens,
                                      B, max_q_len, Hq, Hkv, D, scale_log2, out, 1, nullptr, stream);
  }
  const int64_t col_tiles = (int64_t(max_q_len) * (Hq / Hkv) + kCols - 1) / kCols;
  return launch_attn<kFull>(fn, q, k_pool, v_pool, num_blocks, block_tables, max_blocks, cu_q, seq_lens, B,
                            Hq, Hkv, D, col_tiles, softmax_scale * 1.4426950408889634f, out,
                            static_cast<unsigned*>(workspace), 0, nullptr, nullptr, 0,
                            static_cast<hipStream_t>(stream));
}


extern "C" int ilpc_decode_split(int32_t B, int32_t Hkv, int32_t max_blocks, int32_t* n_split) {
  if (!n_split || B < 0 || Hkv < 1 || max_blocks < 1)
    return ilpc::set_error(ILPC_EINVAL, "ilpc_decode_split: bad argument");
  *n_split = decode_auto_split(B, Hkv, max_blocks);
  return ILPC_OK;
}

extern "C" int ilpc_decode_workspace_bytes(int32_t B, int32_t max_q_len, int32_t Hq, int32_t Hkv, int32_t D,
                                           int32_t n_split, size_t* bytes) {
  if (!bytes || B < 0 || max_q_len < 0 || Hq < 1 || Hkv < 1 || D < 1 || n_split < 1 ||
      n_split > ilpc::kMaxSplit)
    return ilpc::set_error(ILPC_EINVAL, "ilpc_decode_workspace_bytes: bad argument");
  *bytes = ilpc::decode_split_bytes(B, max_q_len, Hq, Hkv, D, n_split);
  return ILPC_OK;
}

extern "C" int ilpc_paged_decode_attn(const uint16_t* q, const uint16_t* k_pool, const uint16_t* v_pool,
                                     int32_t num_blocks, const int32_t* block_tables, int32_t max_blocks,
                                     const int32_t* cu_q, const int32_t* seq_lens, int32_t B, int32_t max_q_len,
                                     int32_t Hq, int32_t Hkv, int32_t D, int32_t block_size,
                                     float softmax_scale, uint16_t* out, int32_t n_split, void* workspace,
                                     size_t workspace_bytes, void* stream) {
  static const char* fn = "ilpc_paged_decode_attn";
  int rc = check_attn_args(fn, q, k_pool, v_pool, num_blocks, block_tables, max_blocks, cu_q, seq_lens, B,
                           max_q_len, Hq, Hkv, D, block_size, softmax_scale, out);
  if (rc != ILPC_OK || B == 0 || max_q_len == 0) return rc;
  if (int64_t(max_q_len) * (Hq / Hkv) > kDecodeCols)
    return ilpc::set_error(ILPC_EUNSUP, "%s: max_q_len * Hq / Hkv = %lld > %d", fn,
                           (long long)max_q_len * (Hq / Hkv), kDecodeCols);
  if (n_split < 0 || n_split > ilpc::kMaxSplit)
    return ilpc::set_error(ILPC_EINVAL, "%s: n_split %d outside [0, %d]", fn, n_split, ilpc::kMaxSplit);
  if (n_split == 0) n_split = decode_auto_split(B, Hkv, max_blocks);
  if (int64_t(B) * Hkv * n_split > INT32_MAX)
    return ilpc::set_error(ILPC_EUNSUP, "%s: B * Hkv * n_split too large", fn);
  const size_t need = ilpc::decode_split_bytes(B, max_q_len, Hq, Hkv, D, n_split);
  if (need && (!workspace || workspace_bytes < need || !aligned16(workspace)))
    return ilpc::set_error(ILPC_EINVAL, "%s: %d key ranges need a %zu-byte workspace, 16-byte aligned", fn,
                           n_split, need);
  return ilpc::launch_decode_attn(q, k_pool, v_pool, num_blocks, block_tables, max_blocks, cu_q, seq_lens, B,
                                  max_q_len, Hq, Hkv, D, softmax_scale * 1.4426950408889634f, out, n_split,
                                  static_cast<float*>(workspace), stream);
}

extern "C" int ilpc_attn_cascade_workspace_bytes(int32_t B, int32_t max_q_len, int32_t Hq, int32_t Hkv,
                                                 int32_t D, size_t* bytes) {
  if (!bytes || B < 0 || max_q_len < 0 || Hq < 1 || Hkv < 1 || D < 1)
    return ilpc::set_error(ILPC_EINVAL, "ilpc_attn_cascade_workspace_bytes: bad argument");
  *bytes = cascade_bytes(int64_t(B) * max_q_len, Hq, D);
  return ILPC_OK;
}

extern "C" int ilpc_paged_prefill_attn_cascade(
    const uint16_t* q, const uint16_t* k_pool, const uint16_t* v_pool, int32_t num_blocks,
    const int32_t* block_tables, int32_t max_blocks, const int32_t* cu_q, const int32_t* seq_lens,
    int32_t B, int32_t max_q_len, int32_t Hq, int32_t Hkv, int32_t D, int32_t block_size,
    int32_t shared_len, float softmax_scale, uint16_t* out, void* workspace, size_t workspace_bytes,
    void* stream) {
  static const char* fn = "ilpc_paged_prefill_attn_cascade";
  int rc = check_attn_args(fn, q, k_pool, v_pool, num_blocks, block_tables, max_blocks, cu_q, seq_lens, B,
                           max_q_len, Hq, Hkv, D, block_size, softmax_scale, out);
  if (rc != ILPC_OK) return rc;
  if (shared_len < 0 || shared_len % kBlock != 0 || shared_len > max_blocks * kBlock)
    return ilpc::set_error(ILPC_EINVAL, "%s: shared_len %d must be a multiple of 16 in [0, 16 * max_blocks]",
                           fn, shared_len);
  if (B == 0 || max_q_len == 0) return ILPC_OK;
  const int64_t rows = int64_t(B) * max_q_len;
  if (rows * Hq > (int64_t(1) << 31) - 1) return ilpc::set_error(ILPC_EUNSUP, "%s: batch too large", fn);
  const size_t need = cascade_bytes(rows, Hq, D);
  if (!workspace || workspace_bytes < need || !aligned16(workspace))
    return ilpc::set_error(ILPC_EINVAL, "%s: workspace must be %zu bytes, 16-byte aligned", fn, need);
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  unsigned* queue_shared = reinterpret_cast<unsigned*>(ws);
  unsigned* queue_suffix = reinterpret_cast<unsigned*>(ws + kQueueWords * sizeof(unsigned));
  float* part_o = reinterpret_cast<float*>(ws + kCascadeHead);
  float* part_ml = reinterpret_cast<float*>(ws + kCascadeHead + cascade_part_o_bytes(rows, Hq, D));
  const float scale_log2 = softmax_scale * 1.4426950408889634f;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int G = Hq / Hkv;
  const int64_t col_tiles = (int64_t(max_q_len) * G + kCols - 1) / kCols;
  if (shared_len == 0)
    return launch_attn<kFull>(fn, q, k_pool, v_pool, num_blocks, block_tables, max_blocks, cu_q, seq_lens,
                              B, Hq, Hkv, D, col_tiles, scale_log2, out, queue_shared, 0, nullptr, nullptr,
                              0, s);
  // One launch (kFused) for prefill-shaped batches whose shared prefix holds
  // at least three 64-key tiles and whose per-item tile list fits: at most
  // 256 / G + 1 requests have rows in an item, each with at most
  // ceil(16 * max_blocks / 64) - T_s tiles of its own.
  const int64_t T_s = shared_len / kKeys;
  const int64_t own_tiles = std::max<int64_t>(0, (int64_t(max_blocks) * kBlock + kKeys - 1) / kKeys - T_s);
  if (T_s >= 3 && int64_t(max_q_len) * G >= 2 * kColsPerWave &&
      ((kCols + G - 1) / G + 1) * own_tiles <= kFusedTiles)
    return launch_attn<kFused>(fn, q, k_pool, v_pool, num_blocks, block_tables, max_blocks, cu_q, seq_lens, B,
                               Hq, Hkv, D, (rows * G + kCols - 1) / kCols, scale_log2, out, queue_shared,
                               int(T_s * kKeys), nullptr, nullptr, int(rows), s);
  rc = launch_attn<kShared>(fn, q, k_pool, v_pool, num_blocks, block_tables, max_blocks, cu_q, seq_lens, B,
                            Hq, Hkv, D, (rows * G + kCols - 1) / kCols, scale_log2, out, queue_shared,
                            shared_len, part_o, part_ml, int(rows), s);
  if (rc != ILPC_OK) return rc;
  return launch_attn<kSuffix>(fn, q, k_pool, v_pool, num_blocks, block_tables, max_blocks, cu_q, seq_lens, B,
                              Hq, Hkv, D, col_tiles, scale_log2, out, queue_suffix, shared_len, part_o,
                              part_ml, int(rows), s);
}
