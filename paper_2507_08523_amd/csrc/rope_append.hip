// Rotary position embedding fused into the paged K/V append, for gfx950.
//
// InferLog section 2.1.2: the cached KV carries each token's position, so a
// prompt's new tokens are rotated at their absolute positions (cached prefix
// length + offset) before their K is stored next to the reused prefix.  The
// LLMs the paper serves (Llama-3, Qwen2.5) rotate with RoPE in the
// "rotate-half" arrangement: dimension i < D/2 pairs with i + D/2, and the
// pair turns by the angle pos * inv_freq[i] (Su et al., RoFormer, 2021).
//
// One workgroup per (logical pool block touched, kv head, request), as for
// the plain append: it rotates the block's new K rows and the same positions'
// query rows of the G = Hq / Hkv heads of that kv head.  The cos/sin of each
// (position, frequency) of the block is computed once into LDS and used for
// 1 + G heads.  K goes to the token-major pool block, V (not rotated) to the
// dimension-major block through LDS, rotated Q to q_out (which may alias q:
// every element is read and written by the same thread).
#include <hip/hip_runtime.h>

#include <cstdint>

#include "../../include/ilpc.h"
#include "ilpc_internal.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 16;
constexpr int kMaxGroup = 64;

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) { return __uint_as_float(bits16 << 16); }

// fp32 -> bf16 bits, round to nearest even (inputs are finite).
__device__ __forceinline__ uint32_t f32_to_bf16(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// Rotates 8 consecutive dimensions `lo` (i .. i+7, i < D/2) and their partners
// `hi` (i+D/2 .. i+D/2+7) of one row: lo' = lo*c - hi*s, hi' = hi*c + lo*s.
__device__ __forceinline__ void rotate8(u32x4& lo, u32x4& hi, const float* c, const float* s) {
  u32x4 olo, ohi;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    uint32_t rl = 0, rh = 0;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const float a = bf16_to_f32((lo[w] >> (16 * e)) & 0xFFFFu);
      const float b = bf16_to_f32((hi[w] >> (16 * e)) & 0xFFFFu);
      const int j = 2 * w + e;
      rl |= f32_to_bf16(a * c[j] - b * s[j]) << (16 * e);
      rh |= f32_to_bf16(b * c[j] + a * s[j]) << (16 * e);
    }
    olo[w] = rl;
    ohi[w] = rh;
  }
  lo = olo;
  hi = ohi;
}

template <int D>
__global__ __launch_bounds__(256) void rope_kv_append_kernel(
    const uint16_t* q, uint16_t* q_out, int Hq, const uint16_t* __restrict__ k_new,
    const uint16_t* __restrict__ v_new, uint16_t* __restrict__ k_pool, uint16_t* __restrict__ v_pool,
    int num_blocks, const int32_t* __restrict__ block_tables, int max_blocks,
    const int32_t* __restrict__ cu_new, const int32_t* __restrict__ start_pos, int max_new, int Hkv,
    const float* __restrict__ inv_freq) {
  constexpr int kHalf = D / 2;
  constexpr int kPairs = kHalf / 8;  // 8-dimension chunk pairs per row
  constexpr int kChunks = D / 8;
  __shared__ __attribute__((aligned(16))) uint16_t sv[kBlock][D + 8];
  __shared__ float scos[kBlock][kHalf], ssin[kBlock][kHalf];
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
  const bool store_kv = phys >= 0 && phys < num_blocks;  // uniform across the workgroup
  const int tid = threadIdx.x;
  const int G = Hq / Hkv;
  const size_t kblk = store_kv ? (size_t(phys) * Hkv + h) * kBlock * D : 0;

  // cos / sin of every (position, frequency) of the block, once; V rows to LDS.
  for (int idx = tid; idx < kBlock * kHalf; idx += 256) {
    const int slot = idx / kHalf, i = idx % kHalf;
    const int p = lb * kBlock + slot;
    if (p >= p0 && p < p1) sincosf(float(p) * inv_freq[i], &ssin[slot][i], &scos[slot][i]);
  }
  if (store_kv) {
    for (int idx = tid; idx < kBlock * kChunks; idx += 256) {
      const int slot = idx / kChunks, c8 = idx % kChunks;
      const int p = lb * kBlock + slot;
      if (p >= p0 && p < p1)
        *(u32x4*)(&sv[slot][c8 * 8]) =
            *(const u32x4*)(v_new + (size_t(row0 + p - start) * Hkv + h) * D + c8 * 8);
    }
  }
  __syncthreads();

  // Rotate: item (slot, chunk pair, head), head G standing for the K row.
  const int n_heads = (q ? G : 0) + (store_kv ? 1 : 0);
  for (int idx = tid; idx < kBlock * kPairs * n_heads; idx += 256) {
    const int hd = idx / (kBlock * kPairs), rem = idx % (kBlock * kPairs);
    const int slot = rem / kPairs, j = rem % kPairs;
    const int p = lb * kBlock + slot;
    if (p < p0 || p >= p1) continue;
    const size_t row = size_t(row0 + p - start);
    float c[8], sn[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      c[e] = scos[slot][j * 8 + e];
      sn[e] = ssin[slot][j * 8 + e];
    }
    const bool is_k = !q || hd == G;
    const uint16_t* src = is_k ? k_new + (row * Hkv + h) * D : q + (row * Hq + size_t(h) * G + hd) * D;
    u32x4 lo = *(const u32x4*)(src + j * 8), hi = *(const u32x4*)(src + kHalf + j * 8);
    rotate8(lo, hi, c, sn);
    uint16_t* dst = is_k ? k_pool + kblk + size_t(slot) * D : q_out + (row * Hq + size_t(h) * G + hd) * D;
    *(u32x4*)(dst + j * 8) = lo;
    *(u32x4*)(dst + kHalf + j * 8) = hi;
  }
  if (!store_kv) return;

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

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

extern "C" int ilpc_rope_kv_append(const uint16_t* q, uint16_t* q_out, int32_t Hq,
                                   const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_pool,
                                   uint16_t* v_pool, int32_t num_blocks, const int32_t* block_tables,
                                   int32_t max_blocks, const int32_t* cu_new, const int32_t* start_pos,
                                   int32_t B, int32_t max_new, int32_t Hkv, int32_t D,
                                   int32_t block_size, const float* inv_freq, void* stream) {
  using ilpc::set_error;
  const char* fn = "ilpc_rope_kv_append";
  if (B < 0 || max_new < 0 || num_blocks < 0 || max_blocks < 1 || Hkv < 1 || Hq < 1)
    return set_error(ILPC_EINVAL, "%s: negative or zero size", fn);
  if (block_size != kBlock) return set_error(ILPC_EUNSUP, "%s: block_size must be 16", fn);
  if (D != 64 && D != 128) return set_error(ILPC_EUNSUP, "%s: head_dim %d unsupported", fn, D);
  if (Hq % Hkv != 0 || Hq / Hkv > kMaxGroup)
    return set_error(ILPC_EUNSUP, "%s: Hq %d / Hkv %d unsupported", fn, Hq, Hkv);
  if ((q == nullptr) != (q_out == nullptr))
    return set_error(ILPC_EINVAL, "%s: q and q_out must both be given or both be NULL", fn);
  if (B == 0 || max_new == 0) return ILPC_OK;
  if (!k_new || !v_new || !k_pool || !v_pool || !block_tables || !cu_new || !start_pos || !inv_freq)
    return set_error(ILPC_EINVAL, "%s: NULL pointer", fn);
  if (!aligned16(k_new) || !aligned16(v_new) || !aligned16(k_pool) || !aligned16(v_pool) ||
      (q && (!aligned16(q) || !aligned16(q_out))))
    return set_error(ILPC_EINVAL, "%s: Q/K/V buffers must be 16-byte aligned", fn);
  if (B > 65535 || Hkv > 65535) return set_error(ILPC_EUNSUP, "%s: grid too large", fn);
  const int slots = (max_new + kBlock - 2) / kBlock + 1;  // blocks a run of max_new can touch
  const dim3 grid(slots, Hkv, B);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (D == 128)
    hipLaunchKernelGGL(rope_kv_append_kernel<128>, grid, dim3(256), 0, s, q, q_out, Hq, k_new, v_new,
                       k_pool, v_pool, num_blocks, block_tables, max_blocks, cu_new, start_pos,
                       max_new, Hkv, inv_freq);
  else
    hipLaunchKernelGGL(rope_kv_append_kernel<64>, grid, dim3(256), 0, s, q, q_out, Hq, k_new, v_new,
                       k_pool, v_pool, num_blocks, block_tables, max_blocks, cu_new, start_pos,
                       max_new, Hkv, inv_freq);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return set_error(ILPC_EHIP, "%s: launch failed: %s", fn, hipGetErrorString(e));
  return ILPC_OK;
}
