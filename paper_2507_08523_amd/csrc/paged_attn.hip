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
//    workgroup (4 waves) owns 128 query columns of one (request, kv head); a
//    column is a (token, q head of the group) pair, so the G heads of a group
//    share every K/V tile.  Per 64-key tile (4 pool blocks, gathered through
//    the block table with 16-byte loads and staged in LDS):
//      S^T = K Q^T   on v_mfma_f32_32x32x16_bf16 (a lane owns one column),
//      online softmax in fp32 on exp2 with the scale folded in,
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
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 16;                    // tokens per pool block
constexpr int kWaves = 4;                     // waves per attention workgroup
constexpr int kThreads = 64 * kWaves;
constexpr int kColsPerWave = 32;              // query columns per wave (MFMA N)
constexpr int kCols = kColsPerWave * kWaves;  // query columns per workgroup
constexpr int kKeys = 64;                     // keys per tile
constexpr int kTileBlocks = kKeys / kBlock;
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
// paged attention: grid (column tiles, kv heads, requests), heaviest tile first.
template <int D>
__global__ __launch_bounds__(kThreads, 2) void paged_attn_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_pool,
    const uint16_t* __restrict__ v_pool, int num_blocks, const int32_t* __restrict__ block_tables,
    int max_blocks, const int32_t* __restrict__ cu_q, const int32_t* __restrict__ seq_lens, int Hq,
    int Hkv, float scale_log2, uint16_t* __restrict__ out) {
  constexpr int kDch = D / 16;         // 16-wide contraction chunks of Q.K^T
  constexpr int kDt = D / 32;          // 32-row output tiles of O^T
  constexpr int kRowBytes = D * 2;     // one K row in LDS
  constexpr int kKch = D / 8;          // 16-byte chunks per K row
  constexpr int kKLoads = kKeys * kKch / kThreads;
  constexpr int kVLoads = kTileBlocks * 2 * D / kThreads;
  constexpr int kVBlockBytes = D * 32;  // one [D][16] V block in LDS
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * kKeys * D * 2];
  uint8_t* const sK = smem;
  uint8_t* const sV = smem + kKeys * D * 2;

  const int r = blockIdx.z, kvh = blockIdx.y;
  const int G = Hq / Hkv;
  const int q0 = cu_q[r];
  const int q_len = cu_q[r + 1] - q0;
  const int n_cols = q_len * G;
  const int col0 = int(gridDim.x - 1 - blockIdx.x) * kCols;
  int L = seq_lens[r];
  if (L > max_blocks * kBlock) L = max_blocks * kBlock;
  if (q_len <= 0 || col0 >= n_cols || q_len > L) return;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
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
  const int wave_pos_max = qstart + min(wave_first + kColsPerWave - 1, n_cols - 1) / G;
  const int wg_pos_max = qstart + min(col0 + kCols - 1, n_cols - 1) / G;
  const int n_tiles = wg_pos_max / kKeys + 1;

  bf16x8 qf[kDch];
#pragma unroll
  for (int kc = 0; kc < kDch; ++kc) qf[kc] = as_bf16x8(*(const u32x4*)(q + qrow + kc * 16 + hh * 8));

  const int32_t* bt = block_tables + size_t(r) * max_blocks;
  u32x4 kreg[kKLoads], vreg[kVLoads];

  auto load_tile = [&](int j0) {
#pragma unroll
    for (int it = 0; it < kKLoads; ++it) {
      const int idx = it * kThreads + tid;
      const int key = idx / kKch, c = idx % kKch;
      const int j = j0 + key;
      const int lb = j >> 4;
      const int phys = lb < max_blocks ? bt[lb] : -1;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (j < L && phys >= 0 && phys < num_blocks)
        v = *(const u32x4*)(k_pool + ((size_t(phys) * Hkv + kvh) * kBlock + (j & 15)) * D + c * 8);
      kreg[it] = v;
    }
#pragma unroll
    for (int it = 0; it < kVLoads; ++it) {
      const int idx = it * kThreads + tid;
      const int kb = idx / (2 * D), rem = idx % (2 * D);
      const int d = rem >> 1, hf = rem & 1;
      const int jb = j0 + kb * kBlock + hf * 8;
      const int lb = jb >> 4;
      const int phys = lb < max_blocks ? bt[lb] : -1;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (jb < L && phys >= 0 && phys < num_blocks) {
        v = *(const u32x4*)(v_pool + ((size_t(phys) * Hkv + kvh) * D + d) * kBlock + hf * 8);
        const int nvalid = L - jb;  // keys past the context are zeroed: P = 0 must not meet NaN
        if (nvalid < 8) {
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const uint32_t keep = (2 * w < nvalid ? 0x0000FFFFu : 0u) |
                                  (2 * w + 1 < nvalid ? 0xFFFF0000u : 0u);
            v[w] &= keep;
          }
        }
      }
      vreg[it] = v;
    }
  };

  auto store_tile = [&]() {
#pragma unroll
    for (int it = 0; it < kKLoads; ++it) {
      const int idx = it * kThreads + tid;
      const int key = idx / kKch, c = idx % kKch;
      const int m = key_row(key);
      *(u32x4*)(sK + m * kRowBytes + ((c ^ (m & 7)) << 4)) = kreg[it];
    }
#pragma unroll
    for (int it = 0; it < kVLoads; ++it) {
      const int idx = it * kThreads + tid;
      const int kb = idx / (2 * D), rem = idx % (2 * D);
      const int d = rem >> 1, hf = rem & 1;
      *(u32x4*)(sV + kb * kVBlockBytes + d * 32 + ((hf ^ ((d >> 2) & 1)) << 4)) = vreg[it];
    }
  };

  f32x16 o[kDt];
#pragma unroll
  for (int dt = 0; dt < kDt; ++dt)
#pragma unroll
    for (int i = 0; i < 16; ++i) o[dt][i] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  load_tile(0);
  for (int kt = 0; kt < n_tiles; ++kt) {
    const int j0 = kt * kKeys;
    __syncthreads();
    store_tile();
    __syncthreads();
    if (kt + 1 < n_tiles) load_tile(j0 + kKeys);
    if (!wave_active || j0 > wave_pos_max) continue;

    // S^T = K Q^T for two 32-key halves of the tile.
    f32x16 s[2];
#pragma unroll
    for (int i = 0; i < 16; ++i) { s[0][i] = 0.f; s[1][i] = 0.f; }
#pragma unroll
    for (int kc = 0; kc < kDch; ++kc) {
      const int c = kc * 2 + hh;
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        const int row = st * 32 + n;
        const bf16x8 a = *(const bf16x8*)(sK + row * kRowBytes + ((c ^ (row & 7)) << 4));
        s[st] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kc], s[st], 0, 0, 0);
      }
    }

    // Online softmax over this lane's column (log2 domain).
    const bool need_mask = j0 + kKeys - 1 > wave_pos_min;
    float x[32];
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        float v = s[st][i] * scale_log2;
        if (need_mask) {
          const int key = j0 + st * 32 + (i >> 3) * 16 + hh * 8 + (i & 7);
          if (key > pos) v = -INFINITY;
        }
        x[st * 16 + i] = v;
      }
    float mloc = x[0];
#pragma unroll
    for (int i = 1; i < 32; ++i) mloc = fmaxf(mloc, x[i]);
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
    const float m_new = fmaxf(m_run, mloc);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    m_run = m_new;
    float psum = 0.f;
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      x[i] = __builtin_amdgcn_exp2f(x[i] - m_new);
      psum += x[i];
    }
    l_run = l_run * alpha + psum;
#pragma unroll
    for (int dt = 0; dt < kDt; ++dt)
#pragma unroll
      for (int i = 0; i < 16; ++i) o[dt][i] *= alpha;

    // O^T += V^T P^T, one 16-key pool block at a time.
#pragma unroll
    for (int kb = 0; kb < kTileBlocks; ++kb) {
      bf16x8 pb;
#pragma unroll
      for (int e = 0; e < 8; ++e) pb[e] = (__bf16)x[kb * 8 + e];
#pragma unroll
      for (int dt = 0; dt < kDt; ++dt) {
        const int d = dt * 32 + n;
        const bf16x8 a =
            *(const bf16x8*)(sV + kb * kVBlockBytes + d * 32 + ((hh ^ ((d >> 2) & 1)) << 4));
        o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb, o[dt], 0, 0, 0);
      }
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
  if (B < 0 || max_q_len < 0 || num_blocks < 0 || max_blocks < 1 || Hq < 1 || Hkv < 1)
    return set_error(ILPC_EINVAL, "ilpc_paged_prefill_attn: negative or zero size");
  if (block_size != kBlock)
    return set_error(ILPC_EUNSUP, "ilpc_paged_prefill_attn: block_size must be 16");
  if (D != 64 && D != 128)
    return set_error(ILPC_EUNSUP, "ilpc_paged_prefill_attn: head_dim %d unsupported", D);
  if (Hq % Hkv != 0 || Hq / Hkv > kMaxGroup)
    return set_error(ILPC_EUNSUP, "ilpc_paged_prefill_attn: Hq %d / Hkv %d unsupported", Hq, Hkv);
  if (!std::isfinite(softmax_scale))
    return set_error(ILPC_EINVAL, "ilpc_paged_prefill_attn: softmax_scale is not finite");
  if (B == 0 || max_q_len == 0) return ILPC_OK;
  if (!q || !k_pool || !v_pool || !block_tables || !cu_q || !seq_lens || !out)
    return set_error(ILPC_EINVAL, "ilpc_paged_prefill_attn: NULL pointer");
  if (!aligned16(q) || !aligned16(k_pool) || !aligned16(v_pool) || !aligned16(out))
    return set_error(ILPC_EINVAL, "ilpc_paged_prefill_attn: Q/K/V/out must be 16-byte aligned");
  const int64_t col_tiles = (int64_t(max_q_len) * (Hq / Hkv) + kCols - 1) / kCols;
  if (B > 65535 || Hkv > 65535 || col_tiles > (int64_t(1) << 31) - 1)
    return set_error(ILPC_EUNSUP, "ilpc_paged_prefill_attn: grid too large");
  const float scale_log2 = softmax_scale * 1.4426950408889634f;
  const dim3 grid(unsigned(col_tiles), Hkv, B);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (D == 128)
    hipLaunchKernelGGL(paged_attn_kernel<128>, grid, dim3(kThreads), 0, s, q, k_pool, v_pool,
                       num_blocks, block_tables, max_blocks, cu_q, seq_lens, Hq, Hkv, scale_log2,
                       out);
  else
    hipLaunchKernelGGL(paged_attn_kernel<64>, grid, dim3(kThreads), 0, s, q, k_pool, v_pool,
                       num_blocks, block_tables, max_blocks, cu_q, seq_lens, Hq, Hkv, scale_log2,
                       out);
  return launch_status("ilpc_paged_prefill_attn");
}
