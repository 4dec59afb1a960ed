// Relational kernels: WHERE masks, PK-FK hash join, stable compaction,
// GROUP BY aggregation.
//
// The WHERE clause becomes a per-row boolean (Table 1, WHERE -> boolean mask);
// instead of carrying the full table through the model as the paper's static
// program does, the mask is compacted into the ascending list of surviving
// row ids so that only survivors reach the transformer (the on-device data
// skipping named as a roadmap item in Section 5).
//
// Compaction is three launches over fixed 2048-row blocks:
//   mask    : 64 rows per wave evaluated into one ballot word, block popcount
//   scan    : exclusive scan of the block counts (one workgroup)
//   scatter : popcount prefix inside the block + block offset -> output slot
// The order of survivors is the row order (stable), independent of timing.
#include "aiq_internal.h"

namespace aiq {

__device__ __forceinline__ int64_t load_int(const void* p, int dt, int64_t i) {
  switch (dt) {
    case AIQ_I8: return static_cast<const int8_t*>(p)[i];
    case AIQ_I16: return static_cast<const int16_t*>(p)[i];
    default: return static_cast<const int32_t*>(p)[i];
  }
}

__device__ __forceinline__ bool eval_atom(const DPred& p, int64_t r) {
  const int64_t v = load_int(p.data, p.dtype, r);
  switch (p.op) {
    case AIQ_LT: return v < p.k;
    case AIQ_LE: return v <= p.k;
    case AIQ_GT: return v > p.k;
    case AIQ_GE: return v >= p.k;
    case AIQ_EQ: return v == p.k;
    case AIQ_NE: return v != p.k;
    default: {
      bool m = false;
      for (int i = 0; i < p.n_set; ++i) m |= (v == static_cast<int64_t>(p.set[i]));
      return m;
    }
  }
}

__device__ __forceinline__ bool eval_all(const DPredList& L, int64_t r) {
  for (int i = 0; i < L.n; ++i)
    if (!eval_atom(L.p[i], r)) return false;
  return true;
}

__device__ __forceinline__ uint32_t hash_slot(int32_t key, int log2cap) {
  return (static_cast<uint32_t>(key) * 0x9E3779B1u) >> (32 - log2cap);
}

// Returns the slot holding `key`, or -1.
__device__ __forceinline__ int32_t hash_find(const HashArgs& h, int32_t key) {
  const uint32_t mask = (1u << h.cap_log2) - 1u;
  uint32_t s = hash_slot(key, h.cap_log2);
  for (uint32_t i = 0; i <= mask; ++i) {
    const int32_t k = h.keys[s];
    if (k == key) return static_cast<int32_t>(s);
    if (k == HASH_EMPTY) return -1;
    s = (s + 1) & mask;
  }
  return -1;
}

__device__ __forceinline__ void set_status(int64_t* ctr, int64_t bits) {
  atomicOr(reinterpret_cast<unsigned long long*>(ctr + C_STATUS), static_cast<unsigned long long>(bits));
}

// ------------------------------------------------------------------ fills

__global__ void k_fill_i32(int32_t* p, int64_t n, int32_t v) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}
__global__ void k_fill_i64(int64_t* p, int64_t n, int64_t v) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

static int grid_for(int64_t n, int threads, int cap = 4096) {
  int64_t g = (n + threads - 1) / threads;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return static_cast<int>(g);
}

hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t s) {
  hipLaunchKernelGGL(k_fill_i32, dim3(grid_for(n, 256)), dim3(256), 0, s, p, n, v);
  return hipGetLastError();
}
hipError_t launch_fill_i64(int64_t* p, int64_t n, int64_t v, hipStream_t s) {
  hipLaunchKernelGGL(k_fill_i64, dim3(grid_for(n, 256)), dim3(256), 0, s, p, n, v);
  return hipGetLastError();
}

// ------------------------------------------------------------------ hash build
// One thread per build row: rows passing the build-side predicates insert
// (key -> payload) by linear probing.  A key already present means the build
// key is not unique among passing rows.

__global__ void k_hash_build(DPredList preds, const void* key_col, int32_t key_dt, const void* pay_col,
                             int32_t pay_dt, int64_t n_rows, HashArgs h, int64_t* ctr) {
  const uint32_t mask = (1u << h.cap_log2) - 1u;
  for (int64_t r = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; r < n_rows;
       r += (int64_t)gridDim.x * blockDim.x) {
    if (!eval_all(preds, r)) continue;
    const int32_t key = static_cast<int32_t>(load_int(key_col, key_dt, r));
    const int32_t pay = static_cast<int32_t>(load_int(pay_col, pay_dt, r));
    if (key == HASH_EMPTY) {  // reserved empty-slot value cannot be stored
      set_status(ctr, AIQ_DEV_HASH_FULL);
      continue;
    }
    uint32_t s = hash_slot(key, h.cap_log2);
    bool done = false;
    for (uint32_t i = 0; i <= mask; ++i) {
      const int32_t prev = atomicCAS(&h.keys[s], HASH_EMPTY, key);
      if (prev == HASH_EMPTY) {
        h.vals[s] = pay;
        done = true;
        break;
      }
      if (prev == key) {
        set_status(ctr, AIQ_DEV_DUP_KEY);
        done = true;
        break;
      }
      s = (s + 1) & mask;
    }
    if (!done) set_status(ctr, AIQ_DEV_HASH_FULL);
  }
}

hipError_t launch_hash_build(const DPredList& preds, const void* key_col, int32_t key_dtype,
                             const void* pay_col, int32_t pay_dtype, int64_t n_rows, HashArgs h,
                             int64_t* ctr, hipStream_t s) {
  hipLaunchKernelGGL(k_hash_build, dim3(grid_for(n_rows, 256)), dim3(256), 0, s, preds, key_col,
                     key_dtype, pay_col, pay_dtype, n_rows, h, ctr);
  return hipGetLastError();
}

// ------------------------------------------------------------------ masks

__device__ __forceinline__ void finish_block_count(int count_wave, int32_t* blk_cnt) {
  __shared__ int wsum[REL_THREADS / 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (lane == 0) wsum[w] = count_wave;
  __syncthreads();
  if (threadIdx.x == 0) {
    int t = 0;
    for (int i = 0; i < REL_THREADS / 64; ++i) t += wsum[i];
    blk_cnt[blockIdx.x] = t;
  }
}

// Row r = base + j*256 + threadIdx.x for j in [0, 8): each (j, wave) pair
// yields the ballot word index block*32 + j*4 + wave.
__global__ __launch_bounds__(REL_THREADS) void k_row_mask(DPredList preds, int64_t n_rows,
                                                          const void* probe_key, int32_t pk_dt,
                                                          HashArgs h, int join, uint64_t* mask,
                                                          int32_t* blk_cnt) {
  const int64_t base = static_cast<int64_t>(blockIdx.x) * REL_ROWS_PER_BLOCK;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int cnt = 0;
#pragma unroll
  for (int j = 0; j < REL_ROWS_PER_THREAD; ++j) {
    const int64_t r = base + j * REL_THREADS + threadIdx.x;
    bool ok = r < n_rows && eval_all(preds, r);
    if (ok && join) ok = hash_find(h, static_cast<int32_t>(load_int(probe_key, pk_dt, r))) >= 0;
    const uint64_t word = __ballot(ok);
    if (lane == 0) mask[blockIdx.x * REL_WORDS_PER_BLOCK + j * 4 + w] = word;
    cnt += __popcll(word);
  }
  finish_block_count(cnt, blk_cnt);
}

hipError_t launch_row_mask(const DPredList& preds, int64_t n_rows, const void* probe_key,
                           int32_t probe_key_dtype, HashArgs h, int join, uint64_t* mask,
                           int32_t* blk_cnt, hipStream_t s) {
  const int64_t nb = (n_rows + REL_ROWS_PER_BLOCK - 1) / REL_ROWS_PER_BLOCK;
  if (nb == 0) return hipSuccess;
  hipLaunchKernelGGL(k_row_mask, dim3(static_cast<unsigned>(nb)), dim3(REL_THREADS), 0, s, preds,
                     n_rows, probe_key, probe_key_dtype, h, join, mask, blk_cnt);
  return hipGetLastError();
}

// Survivor i is kept when its label is 1 (the strict yes > no decision).
__global__ __launch_bounds__(REL_THREADS) void k_label_mask(const int32_t* label, const int64_t* n_ptr,
                                                            uint64_t* mask, int32_t* blk_cnt) {
  const int64_t n = *n_ptr;
  const int64_t base = static_cast<int64_t>(blockIdx.x) * REL_ROWS_PER_BLOCK;
  if (base >= n) {
    if (threadIdx.x == 0) blk_cnt[blockIdx.x] = 0;
    return;
  }
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int cnt = 0;
#pragma unroll
  for (int j = 0; j < REL_ROWS_PER_THREAD; ++j) {
    const int64_t i = base + j * REL_THREADS + threadIdx.x;
    const bool ok = i < n && label[i] == 1;
    const uint64_t word = __ballot(ok);
    if (lane == 0) mask[blockIdx.x * REL_WORDS_PER_BLOCK + j * 4 + w] = word;
    cnt += __popcll(word);
  }
  finish_block_count(cnt, blk_cnt);
}

hipError_t launch_label_mask(const int32_t* label, const int64_t* n_ptr, int64_t n_ub,
                             uint64_t* mask, int32_t* blk_cnt, hipStream_t s) {
  const int64_t nb = (n_ub + REL_ROWS_PER_BLOCK - 1) / REL_ROWS_PER_BLOCK;
  if (nb == 0) return hipSuccess;
  hipLaunchKernelGGL(k_label_mask, dim3(static_cast<unsigned>(nb)), dim3(REL_THREADS), 0, s, label,
                     n_ptr, mask, blk_cnt);
  return hipGetLastError();
}

// ------------------------------------------------------------------ scan of block counts
// One workgroup of 1024 threads walks the block counts in tiles of 1024 with a
// running carry.  blk_off[b] = sum of counts of blocks < b; blk_off[nb] = total.

__device__ __forceinline__ int64_t block_exclusive_scan_1024(int64_t v, int64_t* total) {
  __shared__ int64_t wsum[16];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int64_t x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int64_t y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[w] = x;
  __syncthreads();
  int64_t before = 0, all = 0;
  for (int i = 0; i < 16; ++i) {
    const int64_t ws = wsum[i];
    if (i < w) before += ws;
    all += ws;
  }
  __syncthreads();
  *total = all;
  return before + x - v;
}

__global__ __launch_bounds__(1024) void k_scan_blocks(const int32_t* blk_cnt, const int64_t* n_ptr,
                                                      int64_t n_ub, int64_t* blk_off,
                                                      int64_t* total_out) {
  const int64_t n = n_ptr ? *n_ptr : n_ub;
  const int64_t nb = (n + REL_ROWS_PER_BLOCK - 1) / REL_ROWS_PER_BLOCK;
  int64_t carry = 0;
  for (int64_t b0 = 0; b0 < nb; b0 += 1024) {
    const int64_t b = b0 + threadIdx.x;
    const int64_t v = b < nb ? blk_cnt[b] : 0;
    int64_t tot;
    const int64_t ex = block_exclusive_scan_1024(v, &tot);
    if (b < nb) blk_off[b] = carry + ex;
    carry += tot;
  }
  if (threadIdx.x == 0) {
    blk_off[nb] = carry;
    *total_out = carry;
  }
}

hipError_t launch_scan_blocks(const int32_t* blk_cnt, const int64_t* n_ptr, int64_t n_ub,
                              int64_t* blk_off, int64_t* total_out, hipStream_t s) {
  hipLaunchKernelGGL(k_scan_blocks, dim3(1), dim3(1024), 0, s, blk_cnt, n_ptr, n_ub, blk_off, total_out);
  return hipGetLastError();
}

// ------------------------------------------------------------------ scatter
// out_ids[pos] = src_ids ? src_ids[r] : r for every set bit r, in row order.
// With a join the build payload of the row's match is written alongside.

__global__ __launch_bounds__(REL_THREADS) void k_scatter_rows(
    const uint64_t* mask, const int64_t* blk_off, const int64_t* n_ptr, int64_t n_ub,
    const int32_t* src_ids, int32_t* out_ids, int64_t out_cap, const void* probe_key, int32_t pk_dt,
    HashArgs h, int join, int32_t* out_payload, int64_t* ctr) {
  const int64_t n = n_ptr ? *n_ptr : n_ub;
  const int64_t base = static_cast<int64_t>(blockIdx.x) * REL_ROWS_PER_BLOCK;
  if (base >= n) return;
  __shared__ uint64_t words[REL_WORDS_PER_BLOCK];
  __shared__ int32_t wpre[REL_WORDS_PER_BLOCK];
  if (threadIdx.x < REL_WORDS_PER_BLOCK) words[threadIdx.x] = mask[blockIdx.x * REL_WORDS_PER_BLOCK + threadIdx.x];
  __syncthreads();
  if (threadIdx.x == 0) {
    int32_t acc = 0;
    for (int i = 0; i < REL_WORDS_PER_BLOCK; ++i) {
      wpre[i] = acc;
      acc += __popcll(words[i]);
    }
  }
  __syncthreads();
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t boff = blk_off[blockIdx.x];
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  bool overflow = false;
#pragma unroll
  for (int j = 0; j < REL_ROWS_PER_THREAD; ++j) {
    const int wi = j * 4 + w;
    const uint64_t word = words[wi];
    if (!((word >> lane) & 1ull)) continue;
    const int64_t r = base + j * REL_THREADS + threadIdx.x;
    const int64_t pos = boff + wpre[wi] + __popcll(word & below);
    if (pos >= out_cap) {
      overflow = true;
      continue;
    }
    out_ids[pos] = src_ids ? src_ids[r] : static_cast<int32_t>(r);
    if (join && out_payload) {
      const int32_t slot = hash_find(h, static_cast<int32_t>(load_int(probe_key, pk_dt, r)));
      out_payload[pos] = slot >= 0 ? h.vals[slot] : 0;
    }
  }
  if (overflow) set_status(ctr, AIQ_DEV_IDS_CAP);
}

hipError_t launch_scatter_rows(const uint64_t* mask, const int64_t* blk_off, const int64_t* n_ptr,
                               int64_t n_ub, const int32_t* src_ids, int32_t* out_ids,
                               int64_t out_cap, const void* probe_key, int32_t probe_key_dtype,
                               HashArgs h, int join, int32_t* out_payload, int64_t* ctr,
                               hipStream_t s) {
  const int64_t nb = (n_ub + REL_ROWS_PER_BLOCK - 1) / REL_ROWS_PER_BLOCK;
  if (nb == 0) return hipSuccess;
  hipLaunchKernelGGL(k_scatter_rows, dim3(static_cast<unsigned>(nb)), dim3(REL_THREADS), 0, s, mask,
                     blk_off, n_ptr, n_ub, src_ids, out_ids, out_cap, probe_key, probe_key_dtype, h,
                     join, out_payload, ctr);
  return hipGetLastError();
}

// ------------------------------------------------------------------ copy ids (argmax: every survivor kept)

__global__ void k_copy_ids(const int32_t* src, const int64_t* n_ptr, int32_t* dst, int64_t cap,
                           int64_t* ctr, int set_kept) {
  const int64_t n = *n_ptr;
  if (set_kept && blockIdx.x == 0 && threadIdx.x == 0) {
    ctr[C_KEPT] = n;
    if (n > cap) set_status(ctr, AIQ_DEV_IDS_CAP);
  }
  const int64_t lim = n < cap ? n : cap;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < lim; i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}

hipError_t launch_copy_ids(const int32_t* src, const int64_t* n_ptr, int64_t n_ub, int32_t* dst,
                           int64_t cap, int64_t* ctr, int set_kept, hipStream_t s) {
  hipLaunchKernelGGL(k_copy_ids, dim3(grid_for(n_ub, 256)), dim3(256), 0, s, src, n_ptr, dst, cap,
                     ctr, set_kept);
  return hipGetLastError();
}

__global__ void k_copy_f32(const float* src, const int64_t* n_ptr, int32_t per_row, float* dst, int64_t cap_rows) {
  const int64_t n = *n_ptr < cap_rows ? *n_ptr : cap_rows;
  const int64_t total = n * per_row;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}

hipError_t launch_copy_f32(const float* src, const int64_t* n_ptr, int64_t n_ub, int32_t per_row,
                           float* dst, int64_t cap_rows, hipStream_t s) {
  hipLaunchKernelGGL(k_copy_f32, dim3(grid_for(n_ub * per_row, 256)), dim3(256), 0, s, src, n_ptr, per_row, dst,
                     cap_rows);
  return hipGetLastError();
}

// ------------------------------------------------------------------ group by
// mode 1: key = key_col[sel[i]], value = label[i], every survivor.
// mode 2: key = payload[i], value 0, survivors with label 1 only.
// bins[2k] = COUNT, bins[2k+1] = SUM.  Keys outside [0, n_keys) are skipped
// and flagged.  Blocks privatise the bins in LDS when they fit (integer sums,
// so the result does not depend on the order of the atomics).

constexpr int GROUP_LDS_KEYS = 4096;

__global__ __launch_bounds__(256) void k_group_acc(const int32_t* sel, const int32_t* label,
                                                   const int32_t* payload, const int64_t* n_ptr,
                                                   const void* key_col, int32_t key_dt, int mode,
                                                   int32_t n_keys, int64_t* bins, int64_t* ctr) {
  __shared__ int32_t lc[GROUP_LDS_KEYS];
  __shared__ int32_t ls[GROUP_LDS_KEYS];
  const bool priv = n_keys <= GROUP_LDS_KEYS;
  if (priv) {
    for (int k = threadIdx.x; k < n_keys; k += blockDim.x) {
      lc[k] = 0;
      ls[k] = 0;
    }
    __syncthreads();
  }
  const int64_t n = *n_ptr;
  bool bad = false;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    int64_t key;
    int32_t val;
    if (mode == 1) {
      key = load_int(key_col, key_dt, sel[i]);
      val = label[i];
    } else {
      if (label[i] != 1) continue;
      key = payload[i];
      val = 0;
    }
    if (key < 0 || key >= n_keys) {
      bad = true;
      continue;
    }
    if (priv) {
      atomicAdd(&lc[key], 1);
      atomicAdd(&ls[key], val);
    } else {
      atomicAdd(reinterpret_cast<unsigned long long*>(&bins[2 * key]), 1ull);
      atomicAdd(reinterpret_cast<unsigned long long*>(&bins[2 * key + 1]),
                static_cast<unsigned long long>(static_cast<int64_t>(val)));
    }
  }
  if (bad) set_status(ctr, AIQ_DEV_GROUP_RANGE);
  if (priv) {
    __syncthreads();
    for (int k = threadIdx.x; k < n_keys; k += blockDim.x) {
      if (lc[k]) {
        atomicAdd(reinterpret_cast<unsigned long long*>(&bins[2 * k]), static_cast<unsigned long long>(lc[k]));
        atomicAdd(reinterpret_cast<unsigned long long*>(&bins[2 * k + 1]),
                  static_cast<unsigned long long>(static_cast<int64_t>(ls[k])));
      }
    }
  }
}

hipError_t launch_group_accumulate(const int32_t* sel, const int32_t* label, const int32_t* payload,
                                   const uint8_t* /*keep_by_label*/, const int64_t* n_ptr, int64_t n_ub,
                                   const void* key_col, int32_t key_dtype, int mode,
                                   int32_t n_keys, int64_t* bins, int64_t* ctr, hipStream_t s) {
  // few blocks: each privatised bin array is merged once
  hipLaunchKernelGGL(k_group_acc, dim3(grid_for(n_ub, 256 * 16, 256)), dim3(256), 0, s, sel, label,
                     payload, n_ptr, key_col, key_dtype, mode, n_keys, bins, ctr);
  return hipGetLastError();
}

// Non-empty groups in ascending key order; AVG = SUM / COUNT in fp64.
__global__ __launch_bounds__(1024) void k_group_emit(const int64_t* bins, int32_t n_keys, int32_t* key_out,
                                                     int64_t* cnt_out, int64_t* sum_out, double* avg_out,
                                                     int64_t cap, int mode, int64_t* ctr) {
  int64_t carry = 0;
  for (int64_t k0 = 0; k0 < n_keys; k0 += 1024) {
    const int64_t k = k0 + threadIdx.x;
    const int64_t c = k < n_keys ? bins[2 * k] : 0;
    int64_t tot;
    const int64_t ex = block_exclusive_scan_1024(c > 0 ? 1 : 0, &tot);
    if (c > 0) {
      const int64_t p = carry + ex;
      if (p < cap) {
        const int64_t sm = bins[2 * k + 1];
        key_out[p] = static_cast<int32_t>(k);
        cnt_out[p] = c;
        sum_out[p] = mode == 1 ? sm : 0;
        avg_out[p] = mode == 1 ? static_cast<double>(sm) / static_cast<double>(c) : 0.0;
      }
    }
    carry += tot;
  }
  if (threadIdx.x == 0) {
    ctr[C_GROUPS] = carry < cap ? carry : cap;
    if (carry > cap) set_status(ctr, AIQ_DEV_GROUP_CAP);
  }
}

hipError_t launch_group_emit(const int64_t* bins, int32_t n_keys, int32_t* key_out,
                             int64_t* cnt_out, int64_t* sum_out, double* avg_out, int64_t cap,
                             int mode, int64_t* ctr, hipStream_t s) {
  hipLaunchKernelGGL(k_group_emit, dim3(1), dim3(1024), 0, s, bins, n_keys, key_out, cnt_out, sum_out,
                     avg_out, cap, mode, ctr);
  return hipGetLastError();
}

// ------------------------------------------------------------------ finalize

__global__ void k_finalize(const int64_t* ctr, int64_t* scalars) {
  const int i = threadIdx.x;
  if (i >= AIQ_N_SCALARS) return;
  int64_t v = 0;
  switch (i) {
    case AIQ_S_SELECTED: v = ctr[C_SEL]; break;
    case AIQ_S_KEPT: v = ctr[C_KEPT]; break;
    case AIQ_S_TOKENS: v = ctr[C_TOK]; break;
    case AIQ_S_STATUS: v = ctr[C_STATUS]; break;
    case AIQ_S_GROUPS: v = ctr[C_GROUPS]; break;
    default: v = 0;
  }
  scalars[i] = v;
}

hipError_t launch_finalize(const int64_t* ctr, int64_t* scalars, hipStream_t s) {
  hipLaunchKernelGGL(k_finalize, dim3(1), dim3(64), 0, s, ctr, scalars);
  return hipGetLastError();
}

}  // namespace aiq
