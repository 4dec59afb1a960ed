// Relational kernels: WHERE masks, PK-FK hash join, stable compaction,
// GROUP BY aggregation.
//
// The WHERE clause becomes a per-row boolean (Table 1, WHERE -> boolean mask);
// instead of carrying the full table through the model as the paper's static
// program does, the mask is compacted into the ascending list of surviving
// row ids so that only survivors reach the transformer (the on-device data
// skipping named as a roadmap item in Section 5).
//
// Compaction runs by default as one launch over 8192-row blocks (k_select_lb:
// masks, the block's survivor list in LDS, a decoupled look-back for the
// totals of earlier blocks, outputs written at their final positions).  The
// three-launch form over blocks of REL_ROWS_PER_BLOCK rows remains:
//   mask    : 64 rows per wave evaluated into one ballot word, block popcount
//   scan    : exclusive scan of the block counts (one workgroup)
//   scatter : popcount prefix inside the block + block offset -> output slot
// In both the order of survivors is the row order (stable), independent of
// timing.  The join's hash table is built in global memory; the one-launch
// form probes a copy of it in LDS when it fits (hashagg.hip rehashes it).
// The dense-key GROUP BY bins live in global memory, privatised in LDS per
// block; GROUP BY over arbitrary keys is in hashagg.hip.
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

// Returns the slot holding `key`, or -1.  The empty-slot value is never a
// stored key (the build refuses it), so a probe with that value matches nothing.
__device__ __forceinline__ int32_t hash_find(const HashArgs& h, int32_t key) {
  if (key == HASH_EMPTY) return -1;
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

// Predicate masks.  A block covers 8192 rows in two passes of 4096; in a pass
// lane l of wave w owns the 16 consecutive rows starting at
// base + pass*4096 + w*1024 + 16l, read with 16-byte loads (one for int8, two
// for int16, four for int32 columns).  The predicates are evaluated column by
// column into a 16-bit result per lane; four neighbouring lanes form one
// 64-row mask word (bit b = row 64*word + b of the block, the natural order
// the compaction reads).  Column data must be 16-byte aligned (the plan
// checks this).

template <typename T>
__device__ __forceinline__ void load16(const T* col, int64_t r0, int64_t n_rows, int32_t (&v)[16]) {
  if (r0 + 16 <= n_rows) {
    constexpr int PER = 16 / sizeof(T);   // values per 16-byte load
#pragma unroll
    for (int q = 0; q < 16 / PER; ++q) {
      const int4 raw = *reinterpret_cast<const int4*>(col + r0 + q * PER);
      const T* e = reinterpret_cast<const T*>(&raw);
#pragma unroll
      for (int k = 0; k < PER; ++k) v[q * PER + k] = static_cast<int32_t>(e[k]);
    }
  } else {
#pragma unroll
    for (int k = 0; k < 16; ++k) v[k] = r0 + k < n_rows ? static_cast<int32_t>(col[r0 + k]) : 0;
  }
}

template <typename T, typename Cmp>
__device__ __forceinline__ uint32_t atom16_op(const T* col, int64_t r0, int64_t n_rows, Cmp cmp) {
  int32_t v[16];
  load16<T>(col, r0, n_rows, v);
  uint32_t bits = 0;
#pragma unroll
  for (int k = 0; k < 16; ++k) bits |= static_cast<uint32_t>(cmp(v[k])) << k;
  return bits;
}

// Column values are at most 32-bit; a constant outside the int32 range
// decides every row alike, so the per-row compare runs in 32 bits.
template <typename T>
__device__ __forceinline__ uint32_t atom16(const DPred& P, int64_t r0, int64_t n_rows) {
  const T* col = static_cast<const T*>(P.data);
  const int64_t k = P.k;
  const bool hi = k > INT32_MAX, lo = k < INT32_MIN;
  const int32_t k32 = hi ? INT32_MAX : (lo ? INT32_MIN : static_cast<int32_t>(k));
  switch (P.op) {
    case AIQ_LT:
      if (hi || lo) return hi ? 0xFFFFu : 0u;
      return atom16_op(col, r0, n_rows, [=](int32_t x) { return x < k32; });
    case AIQ_LE:
      if (hi || lo) return hi ? 0xFFFFu : 0u;
      return atom16_op(col, r0, n_rows, [=](int32_t x) { return x <= k32; });
    case AIQ_GT:
      if (hi || lo) return lo ? 0xFFFFu : 0u;
      return atom16_op(col, r0, n_rows, [=](int32_t x) { return x > k32; });
    case AIQ_GE:
      if (hi || lo) return lo ? 0xFFFFu : 0u;
      return atom16_op(col, r0, n_rows, [=](int32_t x) { return x >= k32; });
    case AIQ_EQ:
      if (hi || lo) return 0u;
      return atom16_op(col, r0, n_rows, [=](int32_t x) { return x == k32; });
    case AIQ_NE:
      if (hi || lo) return 0xFFFFu;
      return atom16_op(col, r0, n_rows, [=](int32_t x) { return x != k32; });
    default:   // IN: set values outside the column's type never match (dropped at plan time)
      return atom16_op(col, r0, n_rows, [&](int32_t x) {
        bool m = false;
        for (int i = 0; i < P.n_set; ++i) m |= (x == P.set[i]);
        return m;
      });
  }
}

// fp32 columns: each value widened to fp64 and compared with the fp64
// constant (IEEE: NaN fails every comparison but NE).
template <typename Cmp>
__device__ __forceinline__ uint32_t atom16f_op(const float* col, int64_t r0, int64_t n_rows, Cmp cmp) {
  float v[16];
  if (r0 + 16 <= n_rows) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float4 f = *reinterpret_cast<const float4*>(col + r0 + 4 * q);
      v[4 * q] = f.x;
      v[4 * q + 1] = f.y;
      v[4 * q + 2] = f.z;
      v[4 * q + 3] = f.w;
    }
  } else {
#pragma unroll
    for (int k = 0; k < 16; ++k) v[k] = r0 + k < n_rows ? col[r0 + k] : 0.f;
  }
  uint32_t bits = 0;
#pragma unroll
  for (int k = 0; k < 16; ++k) bits |= static_cast<uint32_t>(cmp(static_cast<double>(v[k]))) << k;
  return bits;
}

__device__ __forceinline__ uint32_t atom16f(const DPred& P, int64_t r0, int64_t n_rows) {
  const float* col = static_cast<const float*>(P.data);
  const double k = P.fk;
  switch (P.op) {
    case AIQ_LT: return atom16f_op(col, r0, n_rows, [=](double x) { return x < k; });
    case AIQ_LE: return atom16f_op(col, r0, n_rows, [=](double x) { return x <= k; });
    case AIQ_GT: return atom16f_op(col, r0, n_rows, [=](double x) { return x > k; });
    case AIQ_GE: return atom16f_op(col, r0, n_rows, [=](double x) { return x >= k; });
    case AIQ_EQ: return atom16f_op(col, r0, n_rows, [=](double x) { return x == k; });
    default: return atom16f_op(col, r0, n_rows, [=](double x) { return x != k; });   // NE (IN rejected at plan)
  }
}

// The mask word of one pass (see above): rows r0 .. r0 + 15 of this lane and
// of the next three lanes; valid in lanes with lane % 4 == 0, whose word goes
// to index pass * 64 + w * 16 + lane / 4 of the block.
__device__ __forceinline__ uint64_t pass_word(const DPredList& preds, int64_t r0, int64_t n_rows,
                                              const void* probe_key, int32_t pk_dt, const HashArgs& h, int join) {
  uint32_t keep = 0;
#pragma unroll
  for (int k = 0; k < 16; ++k) keep |= static_cast<uint32_t>(r0 + k < n_rows) << k;
  for (int i = 0; i < preds.n; ++i) {   // uniform over the grid
    const DPred& P = preds.p[i];
    if (P.dtype == AIQ_I8) keep &= atom16<int8_t>(P, r0, n_rows);
    else if (P.dtype == AIQ_I16) keep &= atom16<int16_t>(P, r0, n_rows);
    else if (P.dtype == AIQ_F32) keep &= atom16f(P, r0, n_rows);
    else keep &= atom16<int32_t>(P, r0, n_rows);
  }
  if (join) {
    for (int k = 0; k < 16; ++k)
      if ((keep >> k) & 1u)
        if (hash_find(h, static_cast<int32_t>(load_int(probe_key, pk_dt, r0 + k))) < 0) keep &= ~(1u << k);
  }
  const uint32_t k1 = __shfl_down(keep, 1), k2 = __shfl_down(keep, 2), k3 = __shfl_down(keep, 3);
  return static_cast<uint64_t>(keep) | (static_cast<uint64_t>(k1) << 16) | (static_cast<uint64_t>(k2) << 32) |
         (static_cast<uint64_t>(k3) << 48);
}

__global__ __launch_bounds__(REL_THREADS) void k_row_mask(DPredList preds, int64_t n_rows,
                                                          const void* probe_key, int32_t pk_dt,
                                                          HashArgs h, int join, uint64_t* mask,
                                                          int32_t* blk_cnt) {
  const int64_t base = static_cast<int64_t>(blockIdx.x) * REL_ROWS_PER_BLOCK;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int cnt = 0;
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    const int64_t r0 = base + pass * 4096 + w * 1024 + lane * 16;
    const uint64_t word = pass_word(preds, r0, n_rows, probe_key, pk_dt, h, join);
    if ((lane & 3) == 0) {
      mask[blockIdx.x * REL_WORDS_PER_BLOCK + pass * 64 + w * 16 + (lane >> 2)] = word;
      cnt += __popcll(word);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o);
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

// ------------------------------------------------------------------ scan of per-block values
// One workgroup of 1024 threads; each thread sums 32 consecutive block values,
// the workgroup scans those sums, so one pass covers 32768 blocks (268M rows)
// with a running carry across passes.  off[b] = sum of values of blocks < b,
// off[nb] = total.

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

template <typename T>
__global__ __launch_bounds__(1024) void k_scan_blocks(const T* val, const int64_t* n_ptr, int64_t n_ub,
                                                      int64_t* off, int64_t* total_out) {
  constexpr int PER = 32;
  const int64_t n = n_ptr ? *n_ptr : n_ub;
  const int64_t nb = (n + REL_ROWS_PER_BLOCK - 1) / REL_ROWS_PER_BLOCK;
  int64_t carry = 0;
  for (int64_t b0 = 0; b0 < nb; b0 += 1024 * PER) {
    const int64_t first = b0 + static_cast<int64_t>(threadIdx.x) * PER;
    int64_t v[PER];
    int64_t sum = 0;
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      v[k] = first + k < nb ? static_cast<int64_t>(val[first + k]) : 0;
      sum += v[k];
    }
    int64_t tot;
    int64_t run = carry + block_exclusive_scan_1024(sum, &tot);
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      if (first + k < nb) off[first + k] = run;
      run += v[k];
    }
    carry += tot;
  }
  if (threadIdx.x == 0) {
    off[nb] = carry;
    *total_out = carry;
  }
}

hipError_t launch_scan_blocks(const int32_t* blk_cnt, const int64_t* n_ptr, int64_t n_ub,
                              int64_t* blk_off, int64_t* total_out, hipStream_t s) {
  hipLaunchKernelGGL(k_scan_blocks<int32_t>, dim3(1), dim3(1024), 0, s, blk_cnt, n_ptr, n_ub, blk_off, total_out);
  return hipGetLastError();
}

hipError_t launch_scan_blocks64(const int64_t* blk_val, const int64_t* n_ptr, int64_t n_ub,
                                int64_t* blk_off, int64_t* total_out, hipStream_t s) {
  hipLaunchKernelGGL(k_scan_blocks<int64_t>, dim3(1), dim3(1024), 0, s, blk_val, n_ptr, n_ub, blk_off, total_out);
  return hipGetLastError();
}

// ------------------------------------------------------------------ scatter
// out_ids[pos] = src_ids ? src_ids[r] : r for every set bit r, in row order.
// With a join the build payload of the row's match is written alongside;
// with lengths each row's token count too, and the block's token sum.
//
// Two levels: each thread drops the row numbers of its set bits into the
// block's dense list in LDS (slot = popcount prefix of the block's mask),
// then the whole block walks that list with consecutive threads on
// consecutive entries, so every read of ids / offsets and every write of
// ids / lengths is coalesced, and a block with few survivors costs one
// round trip.

__global__ __launch_bounds__(REL_THREADS) void k_scatter_rows(
    const uint64_t* mask, const int64_t* blk_off, const int64_t* n_ptr, int64_t n_ub,
    const int32_t* src_ids, int32_t* out_ids, int64_t out_cap, int32_t* out_ids2, int64_t out_cap2,
    const void* probe_key, int32_t pk_dt, HashArgs h, int join, int32_t* out_payload, ScatterLens ln,
    int64_t* ctr) {
  const int64_t n = n_ptr ? *n_ptr : n_ub;
  const int64_t base = static_cast<int64_t>(blockIdx.x) * REL_ROWS_PER_BLOCK;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (base >= n) {
    if (ln.off && threadIdx.x == 0) ln.blk_tok[blockIdx.x] = 0;
    return;
  }
  __shared__ uint64_t words[REL_WORDS_PER_BLOCK];
  __shared__ int32_t wpre[REL_WORDS_PER_BLOCK + 1];
  __shared__ int32_t wtot;
  __shared__ uint16_t rows[REL_ROWS_PER_BLOCK];   // block-relative row of each survivor, in order
  __shared__ int64_t tsum[REL_THREADS / 64];
  const int64_t boff = blk_off[blockIdx.x];   // issued together with the mask load
  // the block's 128 words and their exclusive popcount prefix (two waves)
  int32_t pc = 0;
  if (threadIdx.x < REL_WORDS_PER_BLOCK) {
    const uint64_t wd = mask[blockIdx.x * REL_WORDS_PER_BLOCK + threadIdx.x];
    words[threadIdx.x] = wd;
    pc = __popcll(wd);
  }
  int32_t x = pc;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int32_t y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (threadIdx.x == 63) wtot = x;
  __syncthreads();
  if (threadIdx.x < REL_WORDS_PER_BLOCK) {
    const int32_t incl = x + (threadIdx.x >= 64 ? wtot : 0);
    wpre[threadIdx.x] = incl - pc;
    if (threadIdx.x == REL_WORDS_PER_BLOCK - 1) wpre[REL_WORDS_PER_BLOCK] = incl;
  }
  __syncthreads();
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
  for (int j = 0; j < REL_ROWS_PER_THREAD; ++j) {
    const int wi = j * 4 + w;
    const uint64_t word = words[wi];
    if ((word >> lane) & 1ull)
      rows[wpre[wi] + __popcll(word & below)] = static_cast<uint16_t>(j * REL_THREADS + threadIdx.x);
  }
  __syncthreads();
  const int32_t cnt = wpre[REL_WORDS_PER_BLOCK];
  bool overflow = false, bad_len = false;
  int64_t tok = 0;
  constexpr int U = 8;   // entries per thread and round, their loads issued together
  for (int i0 = 0; i0 < cnt; i0 += REL_THREADS * U) {
    int32_t id[U];
    uint32_t lo0[U], lo1[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = i0 + u * REL_THREADS + threadIdx.x;
      id[u] = 0;
      lo0[u] = lo1[u] = 0;
      if (i < cnt) {
        const int64_t r = base + rows[i];
        id[u] = src_ids ? src_ids[r] : static_cast<int32_t>(r);
        if (ln.off) {
          // list length from the low 32 bits of both offsets (exact below 2^31)
          const uint32_t* off32 = reinterpret_cast<const uint32_t*>(ln.off);
          lo0[u] = off32[2 * r];
          lo1[u] = off32[2 * r + 2];
        }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = i0 + u * REL_THREADS + threadIdx.x;
      if (i >= cnt) continue;
      const int64_t pos = boff + i;
      if (pos < out_cap) out_ids[pos] = id[u];
      else overflow = true;
      if (out_ids2) {
        if (pos < out_cap2) out_ids2[pos] = id[u];
        else overflow = true;
      }
      if (ln.off) {
        int32_t len = static_cast<int32_t>(lo1[u] - lo0[u]);
        if (len < 0 || len > ln.max_len) {
          bad_len = true;
          len = len < 0 ? 0 : ln.max_len;
        }
        const int32_t l = len + ln.n_prefix;
        ln.lens[pos] = l;
        tok += l;
      }
    }
  }
  if (join && out_payload) {   // the build payload of each survivor's match
    for (int i = threadIdx.x; i < cnt; i += REL_THREADS) {
      const int64_t r = base + rows[i];
      const int32_t slot = hash_find(h, static_cast<int32_t>(load_int(probe_key, pk_dt, r)));
      out_payload[boff + i] = slot >= 0 ? h.vals[slot] : 0;
    }
  }
  if (overflow) set_status(ctr, AIQ_DEV_IDS_CAP);
  if (ln.off) {
    if (bad_len) set_status(ctr, AIQ_DEV_LIST_LEN);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) tok += __shfl_xor(tok, o);
    if (lane == 0) tsum[w] = tok;
    __syncthreads();
    if (threadIdx.x == 0) ln.blk_tok[blockIdx.x] = (tsum[0] + tsum[1]) + (tsum[2] + tsum[3]);
  }
}

hipError_t launch_scatter_rows(const uint64_t* mask, const int64_t* blk_off, const int64_t* n_ptr,
                               int64_t n_ub, const int32_t* src_ids, int32_t* out_ids,
                               int64_t out_cap, const void* probe_key, int32_t probe_key_dtype,
                               HashArgs h, int join, int32_t* out_payload, int64_t* ctr,
                               hipStream_t s, int32_t* out_ids2, int64_t out_cap2, ScatterLens lens) {
  const int64_t nb = (n_ub + REL_ROWS_PER_BLOCK - 1) / REL_ROWS_PER_BLOCK;
  if (nb == 0) return hipSuccess;
  hipLaunchKernelGGL(k_scatter_rows, dim3(static_cast<unsigned>(nb)), dim3(REL_THREADS), 0, s, mask,
                     blk_off, n_ptr, n_ub, src_ids, out_ids, out_cap, out_ids2, out_cap2, probe_key,
                     probe_key_dtype, h, join, out_payload, lens, ctr);
  return hipGetLastError();
}

// ------------------------------------------------------------------ cu_seqlens
// Block b of the compaction owns output positions [blk_off[b], blk_off[b+1]);
// its tokens start at tok_off[b].  Each workgroup writes the exclusive prefix
// cu[i] for its positions, scanning in steps of 4096 (16 per thread, read as
// four 16-byte vectors from an 8-aligned start, written as eight 16-byte
// vectors) with a running carry; the last block also writes cu[n] = total.
// `lens` must be readable up to 23 entries past the last position.
__global__ __launch_bounds__(256) void k_cu_from_blocks(const int32_t* lens, const int64_t* blk_off,
                                                        const int64_t* tok_off, int64_t* cu) {
  constexpr int E = 16;   // entries per thread and step
  __shared__ int64_t wsum[4];
  const int64_t o0 = blk_off[blockIdx.x], o1 = blk_off[blockIdx.x + 1];
  if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) cu[o1] = tok_off[gridDim.x];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int64_t carry = tok_off[blockIdx.x];
  for (int64_t c0 = o0 & ~int64_t(7); c0 < o1; c0 += 256 * E) {
    const int64_t i0 = c0 + static_cast<int64_t>(threadIdx.x) * E;
    int32_t v[E];
    int64_t sum = 0;
    if (i0 < o1) {
#pragma unroll
      for (int q = 0; q < E / 4; ++q) {
        const int4 a = *reinterpret_cast<const int4*>(lens + i0 + 4 * q);
        v[4 * q] = a.x;
        v[4 * q + 1] = a.y;
        v[4 * q + 2] = a.z;
        v[4 * q + 3] = a.w;
      }
#pragma unroll
      for (int k = 0; k < E; ++k) {
        if (!(i0 + k >= o0 && i0 + k < o1)) v[k] = 0;
        sum += v[k];
      }
    } else {
#pragma unroll
      for (int k = 0; k < E; ++k) v[k] = 0;
    }
    int64_t x = sum;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int64_t y = __shfl_up(x, o);
      if (lane >= o) x += y;
    }
    if (lane == 63) wsum[w] = x;
    __syncthreads();
    int64_t before = 0, all = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (i < w) before += wsum[i];
      all += wsum[i];
    }
    __syncthreads();
    int64_t run = carry + before + x - sum;
    if (i0 >= o0 && i0 + E <= o1) {
#pragma unroll
      for (int k = 0; k < E; k += 2) {
        const int64_t a = run;
        run += v[k];
        const int64_t b = run;
        run += v[k + 1];
        *reinterpret_cast<longlong2*>(cu + i0 + k) = make_longlong2(a, b);
      }
    } else {
#pragma unroll
      for (int k = 0; k < E; ++k) {
        if (i0 + k >= o0 && i0 + k < o1) cu[i0 + k] = run;
        run += v[k];
      }
    }
    carry += all;
  }
}

hipError_t launch_cu_from_blocks(const int32_t* lens, const int64_t* blk_off, const int64_t* tok_off,
                                 int64_t n_ub, int64_t* cu, hipStream_t s) {
  const int64_t nb = (n_ub + REL_ROWS_PER_BLOCK - 1) / REL_ROWS_PER_BLOCK;
  if (nb == 0) return launch_fill_i64(cu, 1, 0, s);   // no rows: cu = {0}
  hipLaunchKernelGGL(k_cu_from_blocks, dim3(static_cast<unsigned>(nb)), dim3(256), 0, s, lens, blk_off, tok_off,
                     cu);
  return hipGetLastError();
}

// ------------------------------------------------------------------ single-pass compaction
// WHERE (+ join) masks, stable compaction and the selected rows' token
// offsets in one launch (decoupled look-back).  Block b (LB_ROWS rows,
// 16 per thread) builds its mask words and survivor list in LDS, reads the
// survivors' list offsets, publishes its survivor count and token sum, and
// finds the totals of all earlier blocks by looking back over the published
// values: a predecessor that has already published its inclusive prefix
// ends the walk, one that has published only its own totals is added and the
// walk goes on.  Outputs are then written at their final positions: ids, join
// payloads and cu[pos] = tokens of all earlier selected rows; the last block
// writes the totals (ctr[C_SEL], ctr[C_TOK], cu[n_selected]).  Each row's
// column values and offsets are read once; nothing per row goes back through
// memory.
//
// A block waits only for lower-numbered blocks.  Workgroups are handed to
// each XCD's dispatcher in increasing order and each dispatcher starts them
// in that order, so a block that is waiting never holds the slot that a
// lower-numbered, not yet started block needs.  The wait is still bounded:
// past LB_SPIN_LIMIT polls the block flags AIQ_DEV_SCAN_WAIT and goes on
// with what it has (outputs then invalid).

constexpr int LB_THREADS = 512;
constexpr int LB_ROWS = 16 * LB_THREADS;       // rows per block, 16 per thread
constexpr int LB_WORDS = LB_ROWS / 64;
constexpr int LB_WAVES = LB_THREADS / 64;
static_assert(LB_ROWS >= LB_MIN_ROWS && LB_ROWS <= REL_ROWS_PER_BLOCK && LB_WORDS <= 128, "look-back block size");
constexpr int64_t LB_SET = static_cast<int64_t>(1ull << 63);   // marks a published word
constexpr int LB_SPIN_LIMIT = 1 << 22;

// token counts stored with one spare slot per 16 entries: thread t's 16
// consecutive entries then start in distinct banks
__device__ __forceinline__ int lb_pad(int i) { return i + (i >> 4); }

// Look-back words of block b at lb + 4b: [0] the block's own totals packed as
// tokens << 14 | count (count <= 8192, tokens < 2^31), [1] the inclusive
// count and [2] the inclusive tokens through the block.  Every word carries
// its own published bit, so no ordering between them is needed (relaxed
// device-scope atomics; no other data passes between blocks).
__device__ __forceinline__ int64_t lb_get(const int64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void lb_put(int64_t* p, int64_t v) {
  __hip_atomic_store(p, v | LB_SET, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ int64_t wave_sum64(int64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// STAGED (joins): the block first copies the rehashed build table into LDS
// when it fits (st.log2_out > 0) and probes it there.
template <bool STAGED>
__global__ __launch_bounds__(LB_THREADS) void k_select_lb(
    DPredList preds, int64_t n_rows, int64_t nb, const void* probe_key, int32_t pk_dt, HashArgs h, int join,
    StagedHash st, int32_t* out_ids, int64_t out_cap, int32_t* out_ids2, int64_t out_cap2, int32_t* out_payload,
    const int64_t* off, int32_t max_len, int32_t n_prefix, int64_t* cu, int64_t* lb, int64_t* ctr) {
  __shared__ int32_t jk[STAGED ? JOIN_LDS_SLOTS : 1];
  __shared__ int32_t jv[STAGED ? JOIN_LDS_SLOTS : 1];
  if (STAGED) {
    const int lg = *st.log2_out;
    if (lg > 0) {
      for (int i = threadIdx.x; i < (1 << lg); i += LB_THREADS) {
        jk[i] = st.keys[i];
        jv[i] = st.vals[i];
      }
      __syncthreads();
      h.keys = jk;   // generic pointers into this block's LDS
      h.vals = jv;
      h.cap_log2 = lg;
    }
  }
  __shared__ uint64_t words[LB_WORDS];
  __shared__ int32_t wpre[LB_WORDS + 1];
  __shared__ int32_t wtot;
  __shared__ uint16_t rows[LB_ROWS];                      // block-relative row of each survivor, in order
  __shared__ int32_t tx[LB_ROWS + LB_ROWS / 16];          // token counts, then their prefix
  __shared__ int64_t red[LB_WAVES];
  __shared__ int32_t tscan[LB_WAVES];
  __shared__ int64_t sb[2];                               // count and tokens of all earlier blocks
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int64_t b = blockIdx.x;
  const int64_t base = b * LB_ROWS;
  // masks of the block's rows into LDS (lane l of wave w: rows w*1024 + 16l ..),
  // then their popcount prefix
  {
    const uint64_t word = pass_word(preds, base + w * 1024 + lane * 16, n_rows, probe_key, pk_dt, h, join);
    if ((lane & 3) == 0) words[w * 16 + (lane >> 2)] = word;
  }
  __syncthreads();
  int32_t pc = 0;
  if (t < LB_WORDS) pc = __popcll(words[t]);
  int32_t x = pc;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int32_t y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (LB_WORDS > 64) {
    if (t == 63) wtot = x;
    __syncthreads();
  }
  if (t < LB_WORDS) {
    const int32_t incl = x + (t >= 64 ? wtot : 0);
    wpre[t] = incl - pc;
    if (t == LB_WORDS - 1) wpre[LB_WORDS] = incl;
  }
  __syncthreads();
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const int wi = j * LB_WAVES + w;   // word of rows 64 wi .. 64 wi + 63; this lane's row is 64 wi + lane
    const uint64_t word = words[wi];
    if ((word >> lane) & 1ull)
      rows[wpre[wi] + __popcll(word & below)] = static_cast<uint16_t>(j * LB_THREADS + t);
  }
  __syncthreads();
  const int32_t cnt = wpre[LB_WORDS];
  // token count of every survivor (list length from the low 32 bits of both
  // offsets, exact below 2^31), eight loads per thread in flight
  int64_t tok = 0;
  if (off) {
    bool bad_len = false;
    const uint32_t* off32 = reinterpret_cast<const uint32_t*>(off);
    constexpr int U = 8;
    for (int i0 = 0; i0 < cnt; i0 += LB_THREADS * U) {
      uint32_t lo0[U], lo1[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = i0 + u * LB_THREADS + t;
        lo0[u] = lo1[u] = 0;
        if (i < cnt) {
          const int64_t r = base + rows[i];
          lo0[u] = off32[2 * r];
          lo1[u] = off32[2 * r + 2];
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = i0 + u * LB_THREADS + t;
        if (i >= cnt) continue;
        int32_t len = static_cast<int32_t>(lo1[u] - lo0[u]);
        if (len < 0 || len > max_len) {
          bad_len = true;
          len = len < 0 ? 0 : max_len;
        }
        tx[lb_pad(i)] = len + n_prefix;
        tok += len + n_prefix;
      }
    }
    if (bad_len) set_status(ctr, AIQ_DEV_LIST_LEN);
    tok = wave_sum64(tok);
    if (lane == 0) red[w] = tok;
  }
  __syncthreads();
  if (off) {
    tok = 0;
#pragma unroll
    for (int i = 0; i < LB_WAVES; ++i) tok += red[i];
  }
  // publish this block's totals: block 0 has no predecessor, so its totals
  // are already its inclusive prefix
  int64_t* me = lb + 4 * b;
  if (t == 0) {
    if (b == 0) {
      lb_put(me + 1, cnt);
      lb_put(me + 2, tok);
    } else {
      lb_put(me, (tok << 14) | cnt);
    }
  }
  // exclusive prefix of the token counts inside the block: thread t owns
  // entries 16t .. 16t + 15, 32-bit sums (the plan bounds a block's tokens
  // below 2^31)
  if (off) {
    const int first = t * 16;
    const int lim = cnt - first < 16 ? cnt - first : 16;
    int32_t own = 0;
    for (int k = 0; k < lim; ++k) own += tx[lb_pad(first + k)];
    int32_t y = own;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int32_t z = __shfl_up(y, o);
      if (lane >= o) y += z;
    }
    if (lane == 63) tscan[w] = y;
    __syncthreads();
    int32_t run = y - own;
    for (int i = 0; i < w; ++i) run += tscan[i];
    for (int k = 0; k < lim; ++k) {
      const int a = lb_pad(first + k);
      const int32_t v = tx[a];
      tx[a] = run;
      run += v;
    }
  }
  // look-back over the predecessors: lane l of wave 0 reads block j - l.
  // When the nearest inclusive prefix is not in reach yet, the leading run of
  // published blocks is consumed and the walk continues behind it.
  if (w == 0) {
    int64_t ec = 0, et = 0;
    if (b > 0) {
      int64_t j = b - 1;
      int spins = 0;
      for (;;) {
        const int64_t idx = j - lane;
        int state = 2;   // 2: inclusive prefix, 1: block totals only, 0: nothing yet
        int64_t vc = 0, vt = 0;
        if (idx >= 0) {   // idx < 0: the empty prefix before block 0
          const int64_t* q = lb + 4 * idx;
          const int64_t ag = lb_get(q), ic = lb_get(q + 1), it = lb_get(q + 2);
          if (ic < 0 && it < 0) {
            vc = ic & ~LB_SET;
            vt = it & ~LB_SET;
          } else if (ag < 0) {
            state = 1;
            vc = ag & 0x3FFF;
            vt = (ag >> 14) & 0x7FFFFFFF;
          } else {
            state = 0;
          }
        }
        const uint64_t incl = __ballot(state == 2), ready = __ballot(state != 0);
        const int p = incl ? __ffsll(static_cast<unsigned long long>(incl)) - 1 : 63;
        const uint64_t need = p == 63 ? ~0ull : ((1ull << (p + 1)) - 1);
        if ((ready & need) == need) {
          ec += wave_sum64(lane <= p ? vc : 0);
          et += wave_sum64(lane <= p ? vt : 0);
          if (incl) break;
          j -= 64;
        } else {
          // lanes below the first unpublished one hold block totals only
          const int q = __ffsll(static_cast<unsigned long long>(~ready)) - 1;
          if (q > 0) {
            ec += wave_sum64(lane < q ? vc : 0);
            et += wave_sum64(lane < q ? vt : 0);
            j -= q;
          } else if (++spins > LB_SPIN_LIMIT) {
            if (lane == 0) set_status(ctr, AIQ_DEV_SCAN_WAIT);
            break;
          } else {
            __builtin_amdgcn_s_sleep(1);
          }
        }
      }
      if (lane == 0) {
        lb_put(me + 1, ec + cnt);
        lb_put(me + 2, et + tok);
      }
    }
    if (lane == 0) {
      sb[0] = ec;
      sb[1] = et;
    }
  }
  __syncthreads();
  const int64_t cb = sb[0], tb = sb[1];
  bool overflow = false;
  for (int i = t; i < cnt; i += LB_THREADS) {
    const int64_t pos = cb + i;
    const int32_t id = static_cast<int32_t>(base + rows[i]);
    if (pos < out_cap) out_ids[pos] = id;
    else overflow = true;
    if (out_ids2) {
      if (pos < out_cap2) out_ids2[pos] = id;
      else overflow = true;
    }
    if (cu) cu[pos] = tb + tx[lb_pad(i)];
  }
  if (join && out_payload) {   // the build payload of each survivor's match
    for (int i = t; i < cnt; i += LB_THREADS) {
      const int64_t r = base + rows[i];
      const int32_t slot = hash_find(h, static_cast<int32_t>(load_int(probe_key, pk_dt, r)));
      out_payload[cb + i] = slot >= 0 ? h.vals[slot] : 0;
    }
  }
  if (overflow) set_status(ctr, AIQ_DEV_IDS_CAP);
  if (b == nb - 1 && t == 0) {
    ctr[C_SEL] = cb + cnt;
    if (off) ctr[C_TOK] = tb + tok;
    if (cu) cu[cb + cnt] = tb + tok;
  }
}

hipError_t launch_select_lb(const DPredList& preds, int64_t n_rows, const void* probe_key, int32_t probe_key_dtype,
                            HashArgs h, int join, const StagedHash* st, int32_t* out_ids, int64_t out_cap,
                            int32_t* out_ids2, int64_t out_cap2, int32_t* out_payload, const int64_t* off,
                            int32_t max_len, int32_t n_prefix, int64_t* cu, int64_t* lb, int64_t* ctr,
                            hipStream_t s) {
  const int64_t nb = (n_rows + LB_ROWS - 1) / LB_ROWS;
  if (!off) cu = nullptr;   // no list column: no offsets to write (cu may also be NULL with one: totals only)
  if (nb == 0) return cu ? launch_fill_i64(cu, 1, 0, s) : hipSuccess;   // no rows: cu = {0}
  hipError_t e = launch_fill_i64(lb, 4 * nb, 0, s);
  if (e != hipSuccess) return e;
  if (join && st)
    hipLaunchKernelGGL(k_select_lb<true>, dim3(static_cast<unsigned>(nb)), dim3(LB_THREADS), 0, s, preds, n_rows,
                       nb, probe_key, probe_key_dtype, h, join, *st, out_ids, out_cap, out_ids2, out_cap2,
                       out_payload, off, max_len, n_prefix, cu, lb, ctr);
  else
    hipLaunchKernelGGL(k_select_lb<false>, dim3(static_cast<unsigned>(nb)), dim3(LB_THREADS), 0, s, preds, n_rows,
                       nb, probe_key, probe_key_dtype, h, join, StagedHash{}, out_ids, out_cap, out_ids2, out_cap2,
                       out_payload, off, max_len, n_prefix, cu, lb, ctr);
  return hipGetLastError();
}

__global__ void k_keep_selected(int64_t* ctr, int64_t cap) {
  const int64_t n = ctr[C_SEL];
  ctr[C_KEPT] = n;
  if (n > cap) set_status(ctr, AIQ_DEV_IDS_CAP);
}

hipError_t launch_keep_selected(int64_t* ctr, int64_t cap, hipStream_t s) {
  hipLaunchKernelGGL(k_keep_selected, dim3(1), dim3(1), 0, s, ctr, cap);
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

__global__ void k_finalize(const int64_t* ctr, int64_t* scalars, int32_t tok_per_row, int32_t seq_ctr) {
  const int i = threadIdx.x;
  if (i >= AIQ_N_SCALARS) return;
  int64_t v = 0;
  switch (i) {
    case AIQ_S_SELECTED: v = ctr[C_SEL]; break;
    case AIQ_S_KEPT: v = ctr[C_KEPT]; break;
    case AIQ_S_TOKENS: v = ctr[C_TOK] + static_cast<int64_t>(tok_per_row) * ctr[seq_ctr]; break;
    case AIQ_S_PAIRS: v = ctr[C_PAIRS]; break;
    case AIQ_S_STATUS: v = ctr[C_STATUS]; break;
    case AIQ_S_GROUPS: v = ctr[C_GROUPS]; break;
    default: v = 0;
  }
  scalars[i] = v;
}

hipError_t launch_finalize(const int64_t* ctr, int64_t* scalars, hipStream_t s, int32_t tok_per_row,
                           int32_t seq_ctr) {
  hipLaunchKernelGGL(k_finalize, dim3(1), dim3(64), 0, s, ctr, scalars, tok_per_row, seq_ctr);
  return hipGetLastError();
}

// ------------------------------------------------------------------ SUM of an fp32 column
// Deterministic fp64 sum: SUM_BLOCKS fixed ranges of the selected rows (a
// function of their count only), each summed by 256 threads in index order
// and combined by a fixed butterfly and the four wave sums in order; the
// partials are then combined the same way by one workgroup.

__device__ __forceinline__ double block_sum_fixed(double v, double* wsum, int nw) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  if (lane == 0) wsum[w] = v;
  __syncthreads();
  double t = 0.0;
  for (int i = 0; i < nw; ++i) t += wsum[i];
  return t;
}

__global__ __launch_bounds__(256) void k_sum_partial(const int32_t* sel, const int32_t* label, const int64_t* n_ptr,
                                                     const float* col, int binary, double* partial) {
  __shared__ double wsum[4];
  const int64_t n = *n_ptr;
  const int64_t chunk = (n + SUM_BLOCKS - 1) / SUM_BLOCKS;
  const int64_t lo = blockIdx.x * chunk;
  const int64_t hi = lo + chunk < n ? lo + chunk : n;
  double acc = 0.0;
  for (int64_t i = lo + threadIdx.x; i < hi; i += 256)
    if (!binary || label[i] == 1) acc += static_cast<double>(col[sel[i]]);
  const double t = block_sum_fixed(acc, wsum, 4);
  if (threadIdx.x == 0) partial[blockIdx.x] = t;
}

__global__ __launch_bounds__(SUM_BLOCKS) void k_sum_final(const double* partial, double* out) {
  __shared__ double wsum[SUM_BLOCKS / 64];
  const double t = block_sum_fixed(partial[threadIdx.x], wsum, SUM_BLOCKS / 64);
  if (threadIdx.x == 0) out[0] = t;
}

hipError_t launch_sum_f32(const int32_t* sel, const int32_t* label, const int64_t* n_ptr, const float* col,
                          int binary, double* partial, double* out, hipStream_t s) {
  hipLaunchKernelGGL(k_sum_partial, dim3(SUM_BLOCKS), dim3(256), 0, s, sel, label, n_ptr, col, binary, partial);
  hipLaunchKernelGGL(k_sum_final, dim3(1), dim3(SUM_BLOCKS), 0, s, partial, out);
  return hipGetLastError();
}

}  // namespace aiq
