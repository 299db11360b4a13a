// Paged attention for decode-shaped batches (a few query rows per request),
// for gfx950.
//
// InferLog section 2.1.2: after the prefill, each generated token attends to
// the cached KV of its whole context.  With one to a few query rows per
// request the work is bound by reading K and V from HBM, not by the matrix
// cores, so this kernel drops the workgroup-shared LDS ring of the prefill
// kernel: every wave owns one (request, kv head) and streams that request's K
// and V blocks straight from the pools into registers, two 16-token pool
// blocks (32 keys) per step, with the next step's loads in flight while the
// current one is computed.  The G query heads of the kv head times the
// request's q_len rows (at most 32 columns) form the N side of the same
// v_mfma_f32_32x32x16_bf16 products as the prefill kernel:
//   S^T = K Q^T  (K rows loaded in a permuted key order, so that the score
//                 accumulators are already laid out as the P^T operand),
//   O^T += V^T P^T  (V blocks are stored dimension-major, so each lane's
//                 operand is 16 contiguous bytes of one V row),
// with the online softmax in fp32 on exp2 (Q^T is kept in LDS, so that two
// steps of K/V fit in the registers).  Each XCD takes a contiguous range of
// requests, all kv heads of each: the (block, kv head) slabs of a pool block
// are adjacent in memory, and an XCD's reads stay within its requests' share
// of the pools.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>

#include "../../include/ilpc.h"
#include "ilpc_internal.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 16;
constexpr int kStepKeys = 32;        // keys per step (two pool blocks)
constexpr int kWavesPerGroup = 4;
constexpr float kLazyRescale = 8.f;  // log2 growth of a column max tolerated before rescaling O

// Key held by MFMA row m of a step: inside every 16 keys the groups [4,8)
// and [8,12) trade places, so that accumulator register e of lane half hh
// holds key (e >> 3) * 16 + 8 * hh + (e & 7), the layout of the P^T operand.
__device__ __forceinline__ int key_of_row(int m) {
  const int grp = (m >> 2) & 3;
  return m + (grp == 1 ? 4 : (grp == 2 ? -4 : 0));
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ float max_across_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

template <int D>
struct StepRegs {
  u32x4 k[D / 16];      // K operand, one per 16-dimension chunk
  u32x4 v[2][D / 32];   // V^T operand, [pool block of the step][32-dimension tile]
};

template <int D>
__global__ __launch_bounds__(64 * kWavesPerGroup, 2) void decode_attn_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_pool,
    const uint16_t* __restrict__ v_pool, int num_blocks, const int32_t* __restrict__ block_tables,
    int max_blocks, const int32_t* __restrict__ cu_q, const int32_t* __restrict__ seq_lens, int n_req,
    int max_q_len, int Hq, int Hkv, float scale_log2, uint16_t* __restrict__ out, int n_split,
    int cols_cap, float* __restrict__ part_o, float* __restrict__ part_ml) {
  constexpr int kDch = D / 16, kDt = D / 32;
  // Each wave's Q^T operand lives in LDS (read once per product), which keeps
  // two steps of K/V loads plus O within the registers of two waves per SIMD.
  __shared__ u32x4 q_lds[kWavesPerGroup][kDch][64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int n = lane & 31, hh = lane >> 5;

  // Group b runs on XCD b % 8 (round-robin dispatch); XCD x takes a
  // contiguous range of groups, and items are numbered request-major (about
  // 5% more bandwidth on 512 distinct 2 K-token contexts than kv-head-major
  // numbering, which keeps one kv head's blocks in one XCD's L2 and is 2-3%
  // faster only when every request reads one shared prefix).
  const unsigned nb = gridDim.x, per = nb >> 3, extra = nb & 7u;
  const unsigned x = blockIdx.x & 7u, i = blockIdx.x >> 3;
  const unsigned group = x * per + min(x, extra) + i;
  const int item = int(group) * kWavesPerGroup + wave;
  if (item >= n_req * Hkv * n_split) return;
  // With n_split > 1 the pair's steps are cut into n_split consecutive ranges,
  // one per wave; each wave leaves its unnormalised O, max and sum in
  // part_o / part_ml for decode_combine_kernel (cols_cap = max_q_len * G columns per split).
  const int sp = item % n_split, pair = item / n_split;
  const int r = pair / Hkv, h = pair % Hkv;
  const int G = Hq / Hkv;

  const int q0 = cu_q[r], q_len = cu_q[r + 1] - q0;
  const int L = min(seq_lens[r], max_blocks * kBlock);
  // rows past max_q_len are not computed (the host bounds max_q_len * G by 32)
  const int n_cols = min(q_len, max_q_len) * G;
  if (q_len <= 0 || q_len > L || n_cols > 32) return;

  // This lane's query column (padding columns repeat the last valid one).
  const bool col_valid = n < n_cols;
  const int colc = col_valid ? n : n_cols - 1;
  const int t = colc / G;
  const int pos = L - q_len + t;  // keys 0 .. pos are visible to this column
  const size_t qrow = (size_t(q0 + t) * Hq + size_t(h) * G + (colc - t * G)) * D;
#pragma unroll
  for (int kc = 0; kc < kDch; ++kc) q_lds[wave][kc][lane] = *(const u32x4*)(q + qrow + kc * 16 + hh * 8);

  const int32_t* bt = block_tables + size_t(r) * max_blocks;
  const int n_blk = (L + kBlock - 1) / kBlock;
  const int n_steps_all = (L + kStepKeys - 1) / kStepKeys;
  const int steps_per = (n_steps_all + n_split - 1) / n_split;
  const int s_begin = min(sp * steps_per, n_steps_all);
  const int n_steps = min(s_begin + steps_per, n_steps_all);  // this wave runs steps s_begin .. n_steps-1
  const int krow = key_of_row(n);  // key of the step this lane's K operand row holds
  const size_t head_off = size_t(h) * kBlock * D;
  const size_t slab = size_t(Hkv) * kBlock * D;

  // Block ids come 64 at a time, one per lane, by vector loads issued a
  // window ahead of use (scalar loads would put a memory round trip, and a
  // wait shared with the LDS reads, in front of every step); a step picks its
  // two ids out with readlane.  Ids past the request's blocks or outside the
  // pool read block 0 (those keys are masked and their V rows zeroed).
  auto load_ids = [&](int window) {
    return bt[min(window * 64 + lane, max_blocks - 1)];
  };
  // Window w lives in ids[w & 1]; the other register receives window w + 1
  // (two named registers and a uniform branch: no copy that would wait for
  // the load in flight).
  int win = (2 * s_begin) >> 6;
  int ids0, ids1;
  if (win & 1) {
    ids1 = load_ids(win);
    ids0 = load_ids(win + 1);
  } else {
    ids0 = load_ids(win);
    ids1 = load_ids(win + 1);
  }
  auto block_id = [&](int lb) {
    const int id = (win & 1) ? __builtin_amdgcn_readlane(ids1, lb & 63) : __builtin_amdgcn_readlane(ids0, lb & 63);
    return (lb < n_blk && id >= 0 && id < num_blocks) ? id : 0;
  };
  auto load = [&](int s, StepRegs<D>& R) {
    if ((2 * s) >> 6 != win) {  // steps run in order: the next window
      if (win & 1) ids1 = load_ids(win + 2);
      else ids0 = load_ids(win + 2);
      ++win;
    }
    const int id0 = block_id(2 * s), id1 = block_id(2 * s + 1);
    const int idk = krow < kBlock ? id0 : id1;
    const uint16_t* ks = k_pool + size_t(idk) * slab + head_off + size_t(krow & 15) * D + hh * 8;
#pragma unroll
    for (int kc = 0; kc < kDch; ++kc) R.k[kc] = *(const u32x4*)(ks + kc * 16);
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const uint16_t* vs = v_pool + size_t(b ? id1 : id0) * slab + head_off + size_t(n) * kBlock + hh * 8;
#pragma unroll
      for (int dt = 0; dt < kDt; ++dt) R.v[b][dt] = *(const u32x4*)(vs + dt * 32 * kBlock);
    }
  };

  f32x16 o[kDt];
#pragma unroll
  for (int dt = 0; dt < kDt; ++dt)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[dt][e] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const int mask_from = L - q_len;  // steps reaching past this key need the causal mask

  auto compute = [&](int s, StepRegs<D>& R) {
    const int j0 = s * kStepKeys;
    f32x16 sc;
#pragma unroll
    for (int e = 0; e < 16; ++e) sc[e] = 0.f;
#pragma unroll
    for (int kc = 0; kc < kDch; ++kc)
      sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(R.k[kc]), as_bf16x8(q_lds[wave][kc][lane]), sc,
                                                  0, 0, 0);
    if (j0 + kStepKeys - 1 > mask_from) {
      // causal mask (keys past pos, which also covers keys >= L), and the V
      // rows of keys >= L zeroed: unwritten pool slots may hold any bits
      const int rel = pos - j0 - hh * 8;
#pragma unroll
      for (int e = 0; e < 16; ++e)
        if ((e >> 3) * 16 + (e & 7) > rel) sc[e] = -INFINITY;
      const int lim = L - j0 - hh * 8;  // keys b * 16 + e of this lane's V operand are valid iff < lim
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int dt = 0; dt < kDt; ++dt)
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const int k0 = b * 16 + 2 * w;
            R.v[b][dt][w] &= (k0 < lim ? 0x0000FFFFu : 0u) | (k0 + 1 < lim ? 0xFFFF0000u : 0u);
          }
    }
    float mx = sc[0];
#pragma unroll
    for (int e = 1; e < 16; ++e) mx = fmaxf(mx, sc[e]);
    mx = max_across_halves(mx) * scale_log2;
    // Lazy rescale: O and the sum are rescaled only when a column max grows
    // by more than 2^8 over the one its exponentials are taken against (the
    // first step always sets it: key 0 is visible to every column).
    if (__ballot(mx > m_run + kLazyRescale)) {
      const float m_new = fmaxf(m_run, mx);
      // (a column with nothing visible yet keeps m = -inf and alpha = 1)
      const float alpha = m_new == m_run ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < kDt; ++dt)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[dt][e] *= alpha;
    }
    bf16x8 pb[2];
    float ls = 0.f;
    // until a column has seen a visible key (possible in a split that starts
    // past key 0) its scores and max are -inf: subtract 0 then, so that exp2
    // gives 0 rather than NaN
    const float m_sub = m_run == -INFINITY ? 0.f : m_run;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[e], scale_log2, -m_sub));
      pb[e >> 3][e & 7] = (__bf16)p;
      ls += p;
    }
    l_run += ls;
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int dt = 0; dt < kDt; ++dt)
        o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(R.v[b][dt]), pb[b], o[dt], 0, 0, 0);
  };

  // Two register sets: the next step's loads fly while the current is computed.
  // The scheduling barriers keep each step's loads after the computation that
  // frees their registers: hoisted, they would need a third register set.
  StepRegs<D> ra, rb;
  int s = s_begin;
  if (s < n_steps) load(s, ra);
  for (; s + 1 < n_steps; s += 2) {
    load(s + 1, rb);
    __builtin_amdgcn_sched_barrier(0);
    compute(s, ra);
    __builtin_amdgcn_sched_barrier(0);
    if (s + 2 < n_steps) load(s + 2, ra);
    __builtin_amdgcn_sched_barrier(0);
    compute(s + 1, rb);
    __builtin_amdgcn_sched_barrier(0);
  }
  if (s < n_steps) compute(s, ra);

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (n_split > 1) {
    // partial state of this (pair, split), valid columns only: O [cols_cap][D]
    // (unnormalised) in part_o, (max, sum) [cols_cap][2] in part_ml
    if (col_valid) {
      const size_t slot = (size_t(pair) * n_split + sp) * size_t(cols_cap) + n;
      float* po = part_o + (slot - n) * D;  // row n of this (pair, split)
#pragma unroll
      for (int dt = 0; dt < kDt; ++dt)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const f32x4 v = {o[dt][g4 * 4], o[dt][g4 * 4 + 1], o[dt][g4 * 4 + 2], o[dt][g4 * 4 + 3]};
          *(f32x4*)(po + size_t(n) * D + dt * 32 + g4 * 8 + hh * 4) = v;
        }
      if (hh == 0) {
        part_ml[slot * 2] = m_run;
        part_ml[slot * 2 + 1] = l_tot;
      }
    }
    return;
  }
  if (col_valid) {
    const float inv = 1.f / l_tot;
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

// Merge of the n_split partial states of one (kv head, request, column):
// one wave each.  Lane k reads split k's (max, sum); with M = max_k m_k and
// w_k = 2^(m_k - M), O = sum_k w_k O_k / sum_k w_k l_k.  Lane l covers
// dimensions l * D/64 .. of O.  Split 0 holds key 0, visible to every
// column, so M is finite; a split that saw no visible key has m = -inf,
// O = 0 and weight 0.
template <int D>
__global__ __launch_bounds__(64 * kWavesPerGroup) void decode_combine_kernel(
    const float* __restrict__ part_o, const float* __restrict__ part_ml, const int32_t* __restrict__ cu_q,
    const int32_t* __restrict__ seq_lens,
    int max_blocks, int n_req, int max_q_len, int Hq, int Hkv, int n_split, int cols_cap,
    uint16_t* __restrict__ out) {
  constexpr int kPer = D / 64;  // dimensions per lane
  typedef float vec_t __attribute__((ext_vector_type(kPer)));
  const int lane = threadIdx.x & 63;
  const int64_t w = int64_t(blockIdx.x) * kWavesPerGroup + (threadIdx.x >> 6);
  const int c = int(w % cols_cap);
  const int pair = int(w / cols_cap);
  if (pair >= n_req * Hkv) return;
  const int r = pair / Hkv, h = pair % Hkv;
  const int G = Hq / Hkv;
  const int q0 = cu_q[r], q_len = cu_q[r + 1] - q0;
  const int L = min(seq_lens[r], max_blocks * kBlock);
  const int n_cols = min(q_len, max_q_len) * G;
  if (q_len <= 0 || q_len > L || n_cols > 32 || c >= n_cols) return;

  // slot of (pair, split k, column c) = (pair * n_split + k) * cols_cap + c
  const size_t slot0 = size_t(pair) * n_split * cols_cap + c;
  float m = -INFINITY, l = 0.f;
  if (lane < n_split) {
    m = part_ml[(slot0 + size_t(lane) * cols_cap) * 2];
    l = part_ml[(slot0 + size_t(lane) * cols_cap) * 2 + 1];
  }
  float mx = m;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
  const float wgt = m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - mx);
  float den = wgt * l;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) den += __shfl_xor(den, off);

  const float* po = part_o + slot0 * D + lane * kPer;
  const size_t chunk = size_t(cols_cap) * D;  // stride between splits
  vec_t acc = {};
  int k = 0;
  for (; k + 4 <= n_split; k += 4) {
    vec_t v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = *(const vec_t*)(po + (k + u) * chunk);
#pragma unroll
    for (int u = 0; u < 4; ++u)
      acc += __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wgt), k + u)) * v[u];
  }
  for (; k < n_split; ++k)
    acc += __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wgt), k)) * *(const vec_t*)(po + k * chunk);

  const int t = c / G;
  uint16_t* orow = out + (size_t(q0 + t) * Hq + size_t(h) * G + (c - t * G)) * D + lane * kPer;
  const float inv = 1.f / den;
#pragma unroll
  for (int e = 0; e < kPer; ++e) orow[e] = __builtin_bit_cast(uint16_t, (__bf16)(acc[e] * inv));
}

}  // namespace

namespace ilpc {

size_t decode_split_bytes(int B, int max_q_len, int Hq, int Hkv, int D, int n_split) {
  const int64_t cols = std::min<int64_t>(int64_t(max_q_len) * (Hq / Hkv), 32);
  return n_split > 1 ? size_t(B) * Hkv * n_split * cols * (D + 2) * sizeof(float) : 0;
}

int launch_decode_attn(const uint16_t* q, const uint16_t* k_pool, const uint16_t* v_pool, int num_blocks,
                       const int32_t* block_tables, int max_blocks, const int32_t* cu_q,
                       const int32_t* seq_lens, int B, int max_q_len, int Hq, int Hkv, int D,
                       float scale_log2, uint16_t* out, int n_split, float* part, void* stream_ptr) {
  hipStream_t stream = static_cast<hipStream_t>(stream_ptr);
  if (n_split < 1 || n_split > kMaxSplit || (n_split > 1 && !part))
    return set_error(ILPC_EINVAL, "decode attention: bad split");
  const int cols_cap = int(std::min<int64_t>(int64_t(max_q_len) * (Hq / Hkv), 32));
  float* part_ml = part ? part + size_t(B) * Hkv * n_split * cols_cap * D : nullptr;
  const int64_t items = int64_t(B) * Hkv * n_split;
  const int64_t groups = (items + kWavesPerGroup - 1) / kWavesPerGroup;
  if (groups > (int64_t(1) << 31) - 1) return set_error(ILPC_EUNSUP, "decode attention: batch too large");
  const dim3 grid{unsigned(groups)}, block{64 * kWavesPerGroup};
  if (D == 128)
    hipLaunchKernelGGL(decode_attn_kernel<128>, grid, block, 0, stream, q, k_pool, v_pool, num_blocks,
                       block_tables, max_blocks, cu_q, seq_lens, B, max_q_len, Hq, Hkv, scale_log2, out,
                       n_split, cols_cap, part, part_ml);
  else
    hipLaunchKernelGGL(decode_attn_kernel<64>, grid, block, 0, stream, q, k_pool, v_pool, num_blocks,
                       block_tables, max_blocks, cu_q, seq_lens, B, max_q_len, Hq, Hkv, scale_log2, out,
                       n_split, cols_cap, part, part_ml);
  hipError_t e = hipGetLastError();
  if (e == hipSuccess && n_split > 1) {
    const dim3 cgrid{unsigned((int64_t(B) * Hkv * cols_cap + kWavesPerGroup - 1) / kWavesPerGroup)};
    if (D == 128)
      hipLaunchKernelGGL(decode_combine_kernel<128>, cgrid, block, 0, stream, part, part_ml, cu_q, seq_lens,
                         max_blocks, B, max_q_len, Hq, Hkv, n_split, cols_cap, out);
    else
      hipLaunchKernelGGL(decode_combine_kernel<64>, cgrid, block, 0, stream, part, part_ml, cu_q, seq_lens,
                         max_blocks, B, max_q_len, Hq, Hkv, n_split, cols_cap, out);
    e = hipGetLastError();
  }
  if (e != hipSuccess)
    return set_error(ILPC_EHIP, "decode attention: launch failed: %s", hipGetErrorString(e));
  return ILPC_OK;
}

}  // namespace ilpc
