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
//  * paged_attn: causal grouped-query attention of the suffix queries.  One
//    workgroup (8 waves, one per CU) owns 256 query columns of one (request,
//    kv head); a column is a (token, q head of the group) pair, so the G heads
//    of a group share every K/V tile.  64-key tiles (4 pool blocks) stream
//    through a 4-tile ring in LDS, filled by direct global-to-LDS loads three
//    tiles ahead of use.  Per tile and wave:
//      S^T = K Q^T   on v_mfma_f32_32x32x16_bf16 (a lane owns one column),
//      causal mask, column max, online softmax in fp32 on exp2 with the scale
//      folded in (O is rescaled only when a column max grows by > 2^8),
//      O^T += V^T P^T on the same MFMA, P taken straight from the S^T
//      accumulators (K rows are staged in a permuted order that makes the
//      accumulator layout of S^T equal the operand layout P^T needs).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "../../include/ilpc.h"
#include "ilpc_internal.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 16;                    // tokens per pool block
constexpr int kWaves = 8;                     // waves per attention workgroup
constexpr int kThreads = 64 * kWaves;
constexpr int kColsPerWave = 32;              // query columns per wave (MFMA N)
constexpr int kCols = kColsPerWave * kWaves;  // query columns per workgroup
constexpr int kKeys = 64;                     // keys per tile
constexpr int kTileBlocks = kKeys / kBlock;
constexpr int kStages = 4;                    // K/V tiles resident in the LDS ring
constexpr int kMaxGroup = 64;                 // largest Hq / Hkv accepted

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

// max of three floats in one instruction (v_max3_f32; the operands come from
// the matrix cores or are -inf, never signalling NaNs, so no quieting is needed)
__device__ __forceinline__ float max3f(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

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
// paged attention.  1-D grid over (column tile, kv head, request) work items,
// heaviest column tile of a (request, kv head) first.  Work items are spread
// so that those sharing one (request, kv head) -- and so the same K/V blocks --
// land on the same XCD (workgroups are dealt round-robin to the 8 XCDs, each
// with its own L2).
//
// K/V tiles stream through a ring of kStages tiles in LDS, filled straight
// from HBM by global_load_lds kStages-1 tiles ahead of use; one barrier per
// tile.  Each wave loads one pool block (its K rows and V rows) per tile.
constexpr int kMaxTableBlocks = 1024;  // block-table width the kernel accepts (16384 tokens)
constexpr float kLazyRescale = 8.f;    // log2 growth of a column max tolerated before rescaling O

// s_waitcnt vmcnt(n) with the other counters left free (n < 16).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 16, "vmcnt immediate");
  __builtin_amdgcn_s_waitcnt(0x0F70 | N);
}

// Workgroup barrier without the memory fence of __syncthreads: the caller
// has already waited for exactly the loads it needs.  The empty asm keeps the
// compiler from moving memory accesses across it.
__device__ __forceinline__ void bare_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <int D>
__global__ __launch_bounds__(kThreads, 1) void paged_attn_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_pool,
    const uint16_t* __restrict__ v_pool, int num_blocks, const int32_t* __restrict__ block_tables,
    int max_blocks, const int32_t* __restrict__ cu_q, const int32_t* __restrict__ seq_lens, int Hq,
    int Hkv, int n_col_tiles, float scale_log2, uint16_t* __restrict__ out) {
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
  __shared__ __attribute__((aligned(16))) uint8_t ring[kStages * kStageBytes];
  __shared__ __attribute__((aligned(16))) int32_t s_ids[kMaxTableBlocks + kTileBlocks];

  // XCD-aware decode of the work item.
  const unsigned n_items = gridDim.x, bid = blockIdx.x;
  const unsigned xcd = bid & 7u, per = n_items >> 3, extra = n_items & 7u;
  const unsigned w = xcd * per + min(xcd, extra) + (bid >> 3);
  const int tile = n_col_tiles - 1 - int(w % unsigned(n_col_tiles));
  const unsigned rest = w / unsigned(n_col_tiles);
  const int kvh = int(rest % unsigned(Hkv));
  const int r = int(rest / unsigned(Hkv));

  const int G = Hq / Hkv;
  const int q0 = cu_q[r];
  const int q_len = cu_q[r + 1] - q0;
  const int n_cols = q_len * G;
  const int col0 = tile * kCols;
  int L = seq_lens[r];
  if (L > max_blocks * kBlock) L = max_blocks * kBlock;
  if (q_len <= 0 || col0 >= n_cols || q_len > L) return;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int n = lane & 31, hh = lane >> 5;
  const int qstart = L - q_len;  // position of the request's first query

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
  const int wave_pos_max = wave_active ? qstart + min(wave_first + kColsPerWave - 1, n_cols - 1) / G : -1;
  const int wg_pos_max = qstart + min(col0 + kCols - 1, n_cols - 1) / G;
  const int n_tiles = wg_pos_max / kKeys + 1;
  const int n_blk_used = (wg_pos_max >> 4) + 1;  // <= ceil(L / 16) <= max_blocks
  const int key_lim = wg_pos_max + 1;            // keys at or past this are masked everywhere

  bf16x8 qf[kDch];
#pragma unroll
  for (int kc = 0; kc < kDch; ++kc) qf[kc] = as_bf16x8(*(const u32x4*)(q + qrow + kc * 16 + hh * 8));
  // Q is in before any tile load is issued, so the waits in the tile loop can
  // count tile loads only.
  wait_vmcnt<0>();
  asm volatile("" ::: "memory");

  // Block ids -> LDS; unusable ids read block 0 instead (stray K rows only
  // meet masked scores, stray V rows past key_lim are zeroed below).
  const int32_t* bt = block_tables + size_t(r) * max_blocks;
  for (int i = tid; i < kMaxTableBlocks + kTileBlocks; i += kThreads) {
    int id = 0;
    if (i < n_blk_used) {
      id = bt[i];
      if (id < 0 || id >= num_blocks) id = 0;
    }
    s_ids[i] = id;
  }

  // This wave's direct loads of a tile: all from pool block wave/2 of the tile.
  // LDS slot (row m, slot p) of a K tile holds chunk k_slot(m, p) of key
  // key_row(m); slot (d, p) of a V block holds half v_slot(d, p) of row d.
  uint32_t koff[kKInsts], voff[kVInsts];
#pragma unroll
  for (int it = 0; it < kKInsts; ++it) {
    const int g = wave * kKInsts + it;
    const int m = g * (1024 / kRowBytes) + lane / kKch;
    koff[it] = uint32_t((key_row(m) & 15) * kRowBytes + k_slot<D>(m, lane % kKch) * 16);
  }
#pragma unroll
  for (int it = 0; it < kVInsts; ++it) {
    const int g = wave * kVInsts + it;
    const int d = (g * 1024 % kVBlockBytes) / 32 + (lane >> 1);
    voff[it] = uint32_t(d * 32 + v_slot(d, lane & 1) * 16);
  }
  const int my_blk = wave >> 1;
  const uint8_t* kbase = reinterpret_cast<const uint8_t*>(k_pool) + size_t(kvh) * kSlabBytes;
  const uint8_t* vbase = reinterpret_cast<const uint8_t*>(v_pool) + size_t(kvh) * kSlabBytes;
  const size_t slab_stride = size_t(Hkv) * kSlabBytes;

  auto issue_tile = [&](int tl) {
    const int id = __builtin_amdgcn_readfirstlane(s_ids[tl * kTileBlocks + my_blk]);
    uint8_t* st = ring + (tl % kStages) * kStageBytes;
    const uint8_t* ksrc = kbase + size_t(id) * slab_stride;
    const uint8_t* vsrc = vbase + size_t(id) * slab_stride;
#pragma unroll
    for (int it = 0; it < kKInsts; ++it) global_to_lds16(ksrc + koff[it], st + (wave * kKInsts + it) * 1024);
#pragma unroll
    for (int it = 0; it < kVInsts; ++it)
      global_to_lds16(vsrc + voff[it], st + kKTileBytes + (wave * kVInsts + it) * 1024);
  };
  // Zero the V rows of keys >= key_lim in a V tile (only the tile crossing it).
  auto zero_v_tail = [&](int j0, uint8_t* sV) {
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
  const bf16x2 ones = {(__bf16)1.f, (__bf16)1.f};

  __syncthreads();  // block ids visible
#pragma unroll
  for (int tl = 0; tl < kStages - 1; ++tl)
    if (tl < n_tiles) issue_tile(tl);

  for (int i = 0; i < n_tiles; ++i) {
    const int j0 = i * kKeys;
    // this wave's loads of tile i have landed (later tiles may stay in flight)
    const int ahead = min(kStages - 2, n_tiles - 1 - i);
    if (ahead >= 2) wait_vmcnt<2 * kLoads>();
    else if (ahead == 1) wait_vmcnt<kLoads>();
    else wait_vmcnt<0>();
    bare_barrier();  // every wave's loads of tile i are in; tile i-1's stage is free
    uint8_t* const sK = ring + (i % kStages) * kStageBytes;
    uint8_t* const sV = sK + kKTileBytes;
    if (j0 + kKeys > key_lim) {
      zero_v_tail(j0, sV);
      __syncthreads();
    }
    if (i + kStages - 1 < n_tiles) issue_tile(i + kStages - 1);
    if (j0 > wave_pos_max) continue;

    // S^T = K Q^T for the two 32-key halves of the tile.
    f32x16 s0, s1;
#pragma unroll
    for (int e = 0; e < 16; ++e) { s0[e] = 0.f; s1[e] = 0.f; }
#pragma unroll
    for (int kc = 0; kc < kDch; ++kc) {
      const int c = kc * 2 + hh;
      const bf16x8 a0 = *(const bf16x8*)(sK + n * kRowBytes + (k_slot<D>(n, c) << 4));
      const bf16x8 a1 = *(const bf16x8*)(sK + (32 + n) * kRowBytes + (k_slot<D>(32 + n, c) << 4));
      s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, qf[kc], s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, qf[kc], s1, 0, 0, 0);
    }

    // Causal mask (only tiles that reach past some column's position).
    if (j0 + kKeys - 1 > wave_pos_min) {
      const int rel = pos - j0 - hh * 8;  // key (e>>3)*16 + (e&7) [+32] is visible iff <= rel
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int k = (e >> 3) * 16 + (e & 7);
        s0[e] = k > rel ? -INFINITY : s0[e];
        s1[e] = k + 32 > rel ? -INFINITY : s1[e];
      }
    }

    // Column max; O is rescaled only when it grew by more than 2^kLazyRescale.
    float mx = max3f(s0[0], s1[0], s0[1]);
    mx = max3f(mx, s1[1], s0[2]);
#pragma unroll
    for (int e = 2; e < 15; ++e) mx = max3f(mx, s1[e], s0[e + 1]);
    mx = max3f(mx, s1[15], mx);
    mx = max_across_halves(mx) * scale_log2;
    if (__ballot(mx > m_used + kLazyRescale)) {
      const float m_new = fmaxf(m_used, mx);
      const float alpha = __builtin_amdgcn_exp2f(m_used - m_new);
      m_used = m_new;
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < kDt; ++dt)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[dt][e] *= alpha;
    }

    // P = exp2(S * scale_log2 - m_used) as bf16; the sum uses the same bf16 values.
    bf16x8 pb[kTileBlocks];
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      pb[e >> 3][e & 7] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(s0[e], scale_log2, -m_used));
      pb[2 + (e >> 3)][e & 7] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(s1[e], scale_log2, -m_used));
    }
#pragma unroll
    for (int b = 0; b < kTileBlocks; ++b)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bf16x2 pr = {pb[b][2 * e], pb[b][2 * e + 1]};
        l_run = __builtin_amdgcn_fdot2_f32_bf16(pr, ones, l_run, false);
      }

    // O^T += V^T P^T, one 16-key pool block at a time.
#pragma unroll
    for (int b = 0; b < kTileBlocks; ++b)
#pragma unroll
      for (int dt = 0; dt < kDt; ++dt) {
        const int d = dt * 32 + n;
        const bf16x8 a = *(const bf16x8*)(sV + b * kVBlockBytes + d * 32 + (v_slot(d, hh) << 4));
        o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[b], o[dt], 0, 0, 0);
      }
  }

  if (!wave_active) return;
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = 1.f / l_tot;
  if (!col_valid) return;
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

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

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

extern "C" int ilpc_attn_workspace_bytes(int32_t B, int32_t max_q_len, int32_t Hq, int32_t Hkv,
                                         int32_t D, size_t* bytes) {
  if (!bytes || B < 0 || max_q_len < 0 || Hq < 1 || Hkv < 1 || D < 1)
    return ilpc::set_error(ILPC_EINVAL, "ilpc_attn_workspace_bytes: bad argument");
  *bytes = 0;
  return ILPC_OK;
}

extern "C" int ilpc_paged_prefill_attn(const uint16_t* q, const uint16_t* k_pool,
                                       const uint16_t* v_pool, int32_t num_blocks,
                                       const int32_t* block_tables, int32_t max_blocks,
                                       const int32_t* cu_q, const int32_t* seq_lens, int32_t B,
                                       int32_t max_q_len, int32_t Hq, int32_t Hkv, int32_t D,
                                       int32_t block_size, float softmax_scale, uint16_t* out,
                                       void* workspace, size_t workspace_bytes, void* stream) {
  using ilpc::set_error;
  (void)workspace;
  (void)workspace_bytes;
  if (B < 0 || max_q_len < 0 || num_blocks < 1 || max_blocks < 1 || Hq < 1 || Hkv < 1)
    return set_error(ILPC_EINVAL, "ilpc_paged_prefill_attn: negative or zero size");
  if (block_size != kBlock)
    return set_error(ILPC_EUNSUP, "ilpc_paged_prefill_attn: block_size must be 16");
  if (D != 64 && D != 128)
    return set_error(ILPC_EUNSUP, "ilpc_paged_prefill_attn: head_dim %d unsupported", D);
  if (Hq % Hkv != 0 || Hq / Hkv > kMaxGroup)
    return set_error(ILPC_EUNSUP, "ilpc_paged_prefill_attn: Hq %d / Hkv %d unsupported", Hq, Hkv);
  if (!std::isfinite(softmax_scale))
    return set_error(ILPC_EINVAL, "ilpc_paged_prefill_attn: softmax_scale is not finite");
  if (max_blocks > kMaxTableBlocks)
    return set_error(ILPC_EUNSUP, "ilpc_paged_prefill_attn: max_blocks %d > %d (contexts up to %d tokens)",
                     max_blocks, kMaxTableBlocks, kMaxTableBlocks * kBlock);
  if (B == 0 || max_q_len == 0) return ILPC_OK;
  if (!q || !k_pool || !v_pool || !block_tables || !cu_q || !seq_lens || !out)
    return set_error(ILPC_EINVAL, "ilpc_paged_prefill_attn: NULL pointer");
  if (!aligned16(q) || !aligned16(k_pool) || !aligned16(v_pool) || !aligned16(out))
    return set_error(ILPC_EINVAL, "ilpc_paged_prefill_attn: Q/K/V/out must be 16-byte aligned");
  const int64_t col_tiles = (int64_t(max_q_len) * (Hq / Hkv) + kCols - 1) / kCols;
  const int64_t items = col_tiles * Hkv * B;
  if (items > (int64_t(1) << 31) - 1)
    return set_error(ILPC_EUNSUP, "ilpc_paged_prefill_attn: grid too large");
  const float scale_log2 = softmax_scale * 1.4426950408889634f;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (D == 128)
    hipLaunchKernelGGL(paged_attn_kernel<128>, dim3(unsigned(items)), dim3(kThreads), 0, s, q, k_pool,
                       v_pool, num_blocks, block_tables, max_blocks, cu_q, seq_lens, Hq, Hkv,
                       int(col_tiles), scale_log2, out);
  else
    hipLaunchKernelGGL(paged_attn_kernel<64>, dim3(unsigned(items)), dim3(kThreads), 0, s, q, k_pool,
                       v_pool, num_blocks, block_tables, max_blocks, cu_q, seq_lens, Hq, Hkv,
                       int(col_tiles), scale_log2, out);
  return launch_status("ilpc_paged_prefill_attn");
}
