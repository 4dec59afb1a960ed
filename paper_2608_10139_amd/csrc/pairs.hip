// Pairs of selected rows classified on their joint text: Q4 of Section 4, a
// self-join on the movie id (A.id = B.id AND A.review_id < B.review_id) whose
// AI_IF reads [A.text, B.text].  Fig. 4 of the paper contrasts its host
// transfers (every pair's text crosses PCIe) with the unified plan; here the
// pairs are enumerated, packed and classified in device memory.
//
// Candidates are numbered ascending by (A, B): the selected rows are sorted
// stably by key (counting sort over the dense key domain), each row's later
// partners are the next rows of its key group, and an exclusive scan of the
// partner counts in row order gives each row's first pair number.
#include "aiq_internal.h"
#include "dev_util.h"

namespace aiq {

static int grid_for(int64_t n, int per_block, int cap) {
  int64_t g = (n + per_block - 1) / per_block;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return static_cast<int>(g);
}

__device__ __forceinline__ int64_t key_at(const void* p, int dt, int64_t i) {
  switch (dt) {
    case AIQ_I8: return static_cast<const int8_t*>(p)[i];
    case AIQ_I16: return static_cast<const int16_t*>(p)[i];
    default: return static_cast<const int32_t*>(p)[i];
  }
}

__device__ __forceinline__ void flag(int64_t* ctr, int64_t bits) {
  atomicOr(reinterpret_cast<unsigned long long*>(ctr + C_STATUS), static_cast<unsigned long long>(bits));
}

// exclusive scan over the 1024 threads of a block; *total = the block sum
__device__ __forceinline__ int64_t scan1024(int64_t v, int64_t* total) {
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
  for (int k = 0; k < 16; ++k) {
    const int64_t ws = wsum[k];
    if (k < w) before += ws;
    all += ws;
  }
  __syncthreads();
  *total = all;
  return before + x - v;
}

// ------------------------------------------------------------------ generic scan
// Blocks of REL_ROWS_PER_BLOCK elements (1024 threads x 8): block sums, their
// exclusive scan (the relational block scan), then each block's local scan.
constexpr int SEG = REL_ROWS_PER_BLOCK;
static_assert(SEG == 1024 * 8, "scan block = 1024 threads x 8 elements");

__global__ __launch_bounds__(1024) void k_seg_sum(const int32_t* v, const int64_t* n_ptr, int64_t n_ub,
                                                  int64_t* bs) {
  const int64_t n = n_ptr ? *n_ptr : n_ub;
  const int64_t base = static_cast<int64_t>(blockIdx.x) * SEG + threadIdx.x * 8;
  int64_t s = 0;
#pragma unroll
  for (int e = 0; e < 8; ++e)
    if (base + e < n) s += v[base + e];
  int64_t tot;
  scan1024(s, &tot);
  if (threadIdx.x == 0) bs[blockIdx.x] = tot;
}

__global__ __launch_bounds__(1024) void k_seg_scan(const int32_t* v, const int64_t* n_ptr, int64_t n_ub,
                                                   const int64_t* boff, int64_t* out) {
  const int64_t n = n_ptr ? *n_ptr : n_ub;
  const int64_t base = static_cast<int64_t>(blockIdx.x) * SEG + threadIdx.x * 8;
  int64_t x[8], s = 0;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    x[e] = base + e < n ? v[base + e] : 0;
    s += x[e];
  }
  int64_t tot;
  int64_t run = boff[blockIdx.x] + scan1024(s, &tot);
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    if (base + e < n) out[base + e] = run;
    run += x[e];
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) out[n] = boff[(n + SEG - 1) / SEG];   // the total
}

hipError_t launch_scan_i32_i64(const int32_t* v, const int64_t* n_ptr, int64_t n_ub, int64_t* out, int64_t* blk,
                               int64_t* total_out, hipStream_t s) {
  const int64_t nb = (n_ub + SEG - 1) / SEG;
  const unsigned g = static_cast<unsigned>(nb < 1 ? 1 : nb);
  int64_t* bs = blk;
  int64_t* boff = blk + nb + 2;
  hipLaunchKernelGGL(k_seg_sum, dim3(g), dim3(1024), 0, s, v, n_ptr, n_ub, bs);
  hipError_t e = launch_scan_blocks64(bs, n_ptr, n_ub, boff, total_out, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_seg_scan, dim3(g), dim3(1024), 0, s, v, n_ptr, n_ub, boff, out);
  return hipGetLastError();
}

// ------------------------------------------------------------------ key histogram
__global__ void k_pair_key_count(const int32_t* sel, const int64_t* n_ptr, const void* key_col, int32_t key_dt,
                                 int32_t n_keys, int32_t* kcount, int64_t* ctr) {
  const int64_t n = *n_ptr;
  bool bad = false;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t k = key_at(key_col, key_dt, sel[i]);
    if (k < 0 || k >= n_keys) bad = true;
    else atomicAdd(kcount + k, 1);
  }
  if (bad) flag(ctr, AIQ_DEV_GROUP_RANGE);
}

hipError_t launch_pair_key_count(const int32_t* sel, const int64_t* n_ptr, int64_t n_ub, const void* key_col,
                                 int32_t key_dt, int32_t n_keys, int32_t* kcount, int64_t* ctr, hipStream_t s) {
  hipLaunchKernelGGL(k_pair_key_count, dim3(grid_for(n_ub, 256, 4096)), dim3(256), 0, s, sel, n_ptr, key_col,
                     key_dt, n_keys, kcount, ctr);
  return hipGetLastError();
}

// ------------------------------------------------------------------ stable rank within key
// One workgroup walks the selected rows in rounds of 1024: a bitonic sort of
// (key, index) in LDS puts each round's rows of a key together in index
// order; a row's rank is the key's count from earlier rounds plus its place
// among the round's rows of that key.
__global__ __launch_bounds__(1024) void k_pair_rank(const int32_t* sel, const int64_t* n_ptr, const void* key_col,
                                                    int32_t key_dt, int32_t n_keys, const int64_t* koff,
                                                    int32_t* rank, int32_t* sorted) {
  __shared__ uint64_t buf[1024];
  __shared__ int32_t fs[1024];
  __shared__ int32_t cur[PAIR_MAX_KEYS];
  const int t = threadIdx.x;
  const int64_t n = *n_ptr;
  for (int k = t; k < n_keys; k += 1024) cur[k] = 0;
  __syncthreads();
  for (int64_t base = 0; base < n; base += 1024) {
    const int64_t i = base + t;
    uint32_t key = static_cast<uint32_t>(n_keys);   // past the end or out of range: sorts last, ignored
    if (i < n) {
      const int64_t k = key_at(key_col, key_dt, sel[i]);
      if (k >= 0 && k < n_keys) key = static_cast<uint32_t>(k);
    }
    buf[t] = (static_cast<uint64_t>(key) << 32) | static_cast<uint32_t>(i < n ? i : 0xFFFFFFFFll);
    __syncthreads();
    for (int size = 2; size <= 1024; size <<= 1) {
      for (int stride = size >> 1; stride > 0; stride >>= 1) {
        const int partner = t ^ stride;
        if (partner > t) {
          const uint64_t a = buf[t], b = buf[partner];
          const bool up = (t & size) == 0;
          if ((a > b) == up) {
            buf[t] = b;
            buf[partner] = a;
          }
        }
        __syncthreads();
      }
    }
    const uint64_t my = buf[t];
    const uint32_t kk = static_cast<uint32_t>(my >> 32);
    const uint32_t ii = static_cast<uint32_t>(my);
    fs[t] = (t == 0 || static_cast<uint32_t>(buf[t - 1] >> 32) != kk) ? t : 0;
    __syncthreads();
    for (int o = 1; o < 1024; o <<= 1) {   // first position of each key run: inclusive max scan
      const int v = t >= o ? fs[t - o] : 0;
      __syncthreads();
      if (v > fs[t]) fs[t] = v;
      __syncthreads();
    }
    const int first = fs[t];
    if (kk < static_cast<uint32_t>(n_keys)) {
      const int32_t r = cur[kk] + (t - first);
      rank[ii] = r;
      sorted[koff[kk] + r] = static_cast<int32_t>(ii);
    }
    __syncthreads();
    const bool last = t == 1023 || static_cast<uint32_t>(buf[t + 1] >> 32) != kk;
    if (last && kk < static_cast<uint32_t>(n_keys)) cur[kk] += t - first + 1;
    __syncthreads();
  }
}

hipError_t launch_pair_rank(const int32_t* sel, const int64_t* n_ptr, const void* key_col, int32_t key_dt,
                            int32_t n_keys, const int64_t* koff, int32_t* rank, int32_t* sorted, hipStream_t s) {
  if (n_keys <= 0 || n_keys > PAIR_MAX_KEYS) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_pair_rank, dim3(1), dim3(1024), 0, s, sel, n_ptr, key_col, key_dt, n_keys, koff, rank,
                     sorted);
  return hipGetLastError();
}

// ------------------------------------------------------------------ partners, numbering, emission
__global__ void k_pair_partners(const int32_t* sel, const int64_t* n_ptr, const void* key_col, int32_t key_dt,
                                int32_t n_keys, const int32_t* kcount, const int32_t* rank, int32_t* cnt) {
  const int64_t n = *n_ptr;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t k = key_at(key_col, key_dt, sel[i]);
    cnt[i] = (k >= 0 && k < n_keys) ? kcount[k] - rank[i] - 1 : 0;
  }
}

hipError_t launch_pair_partners(const int32_t* sel, const int64_t* n_ptr, int64_t n_ub, const void* key_col,
                                int32_t key_dt, int32_t n_keys, const int32_t* kcount, const int32_t* rank,
                                int32_t* cnt, hipStream_t s) {
  hipLaunchKernelGGL(k_pair_partners, dim3(grid_for(n_ub, 256, 4096)), dim3(256), 0, s, sel, n_ptr, key_col,
                     key_dt, n_keys, kcount, rank, cnt);
  return hipGetLastError();
}

__global__ void k_pair_total(const int64_t* total, int64_t cap, int64_t* ctr) {
  const int64_t p = *total;
  ctr[C_PAIRS] = p < cap ? p : cap;
  if (p > cap) ctr[C_STATUS] |= AIQ_DEV_PAIR_CAP;
}

hipError_t launch_pair_total(const int64_t* total, int64_t cap, int64_t* ctr, hipStream_t s) {
  hipLaunchKernelGGL(k_pair_total, dim3(1), dim3(1), 0, s, total, cap, ctr);
  return hipGetLastError();
}

// wave per selected row: its partners are the next rows of its key group
__global__ __launch_bounds__(256) void k_pair_emit(const int32_t* sel, const int64_t* n_ptr, const void* key_col,
                                                   int32_t key_dt, int32_t n_keys, const int64_t* koff,
                                                   const int32_t* rank, const int32_t* sorted, const int32_t* cnt,
                                                   const int64_t* poff, int64_t cap, int32_t* pa, int32_t* pb) {
  const int64_t n = *n_ptr;
  const int lane = threadIdx.x & 63;
  const int64_t wave = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6;
  const int64_t n_waves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t i = wave; i < n; i += n_waves) {
    const int32_t c = cnt[i];
    if (c <= 0) continue;
    const int64_t k = key_at(key_col, key_dt, sel[i]);   // in range: c > 0
    const int64_t q0 = poff[i];
    if (q0 >= cap) continue;
    const int64_t p0 = koff[k] + rank[i] + 1;
    for (int64_t t = lane; t < c && q0 + t < cap; t += 64) {
      pa[q0 + t] = static_cast<int32_t>(i);
      pb[q0 + t] = sorted[p0 + t];
    }
  }
}

hipError_t launch_pair_emit(const int32_t* sel, const int64_t* n_ptr, int64_t n_ub, const void* key_col,
                            int32_t key_dt, int32_t n_keys, const int64_t* koff, const int32_t* rank,
                            const int32_t* sorted, const int32_t* cnt, const int64_t* poff, int64_t cap,
                            int32_t* pa, int32_t* pb, hipStream_t s) {
  hipLaunchKernelGGL(k_pair_emit, dim3(grid_for(n_ub, 4, 8192)), dim3(256), 0, s, sel, n_ptr, key_col, key_dt,
                     n_keys, koff, rank, sorted, cnt, poff, cap, pa, pb);
  return hipGetLastError();
}

// ------------------------------------------------------------------ pair sequences
__device__ __forceinline__ int32_t list_len(const int64_t* off, int32_t row, int32_t max_len, bool& bad) {
  int64_t l = off[row + 1] - off[row];
  if (l < 0 || l > max_len) {
    bad = true;
    l = l < 0 ? 0 : max_len;
  }
  return static_cast<int32_t>(l);
}

__global__ void k_pair_lens(const int32_t* pa, const int32_t* pb, const int32_t* sel, const int64_t* off,
                            int32_t max_len, int32_t n_prefix, int32_t* lens, int64_t* ctr) {
  const int64_t P = ctr[C_PAIRS];
  bool bad = false;
  for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < P; q += (int64_t)gridDim.x * blockDim.x)
    lens[q] = n_prefix + list_len(off, sel[pa[q]], max_len, bad) + list_len(off, sel[pb[q]], max_len, bad);
  if (bad) flag(ctr, AIQ_DEV_LIST_LEN);
}

hipError_t launch_pair_lens(const int32_t* pa, const int32_t* pb, const int32_t* sel, const int64_t* off,
                            int32_t max_len, int32_t n_prefix, int64_t cap, int32_t* lens, int64_t* ctr,
                            hipStream_t s) {
  hipLaunchKernelGGL(k_pair_lens, dim3(grid_for(cap, 256, 4096)), dim3(256), 0, s, pa, pb, sel, off, max_len,
                     n_prefix, lens, ctr);
  return hipGetLastError();
}

// wave per pair: prefix, A's tokens, B's tokens (ids outside [0, vocab)
// flagged and replaced by 0, as for single rows)
__global__ __launch_bounds__(256) void k_pair_gather(const int32_t* pa, const int32_t* pb, const int32_t* sel,
                                                     const int64_t* off, const int32_t* tokens, const int64_t* cu,
                                                     Prefix pre, int32_t max_len, int32_t vocab, int64_t t_ub,
                                                     int32_t* packed, int64_t* ctr) {
  const int64_t P = ctr[C_PAIRS];
  const int lane = threadIdx.x & 63;
  const int64_t wave = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6;
  const int64_t n_waves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  bool bad = false, bad_len = false;
  for (int64_t q = wave; q < P; q += n_waves) {
    const int64_t c0 = cu[q], c1 = cu[q + 1];
    if (c1 > t_ub) {   // more tokens than the workspace holds: never written
      bad = true;
      continue;
    }
    int32_t* dst = packed + c0;
    for (int j = lane; j < pre.n; j += 64) dst[j] = pre.tok[j];
    dst += pre.n;
    for (int side = 0; side < 2; ++side) {
      const int32_t row = sel[side == 0 ? pa[q] : pb[q]];
      const int32_t L = list_len(off, row, max_len, bad_len);
      const int32_t* src = tokens + off[row];
      for (int j = lane; j < L; j += 64) {
        int32_t tk = src[j];
        if (tk < 0 || tk >= vocab) {
          bad = true;
          tk = 0;
        }
        dst[j] = tk;
      }
      dst += L;
    }
  }
  if (bad) flag(ctr, AIQ_DEV_TOKEN_RANGE);
  if (bad_len) flag(ctr, AIQ_DEV_LIST_LEN);
}

hipError_t launch_pair_gather(const int32_t* pa, const int32_t* pb, const int32_t* sel, const int64_t* off,
                              const int32_t* tokens, const int64_t* cu, const Prefix& prefix, int32_t max_len,
                              int32_t vocab, int64_t t_ub, int64_t cap, int32_t* packed, int64_t* ctr,
                              hipStream_t s) {
  hipLaunchKernelGGL(k_pair_gather, dim3(grid_for(cap, 4, 8192)), dim3(256), 0, s, pa, pb, sel, off, tokens, cu,
                     prefix, max_len, vocab, t_ub, packed, ctr);
  return hipGetLastError();
}

__global__ void k_pair_rows(const int32_t* ids, const int64_t* n_ptr, const int32_t* pa, const int32_t* pb,
                            const int32_t* sel, int32_t* out_a, int32_t* out_b, int64_t cap) {
  int64_t n = *n_ptr;
  if (n > cap) n = cap;
  for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < n; j += (int64_t)gridDim.x * blockDim.x) {
    const int64_t q = ids ? ids[j] : j;
    if (out_a) out_a[j] = sel[pa[q]];
    if (out_b) out_b[j] = sel[pb[q]];
  }
}

hipError_t launch_pair_rows(const int32_t* ids, const int64_t* n_ptr, int64_t n_ub, const int32_t* pa,
                            const int32_t* pb, const int32_t* sel, int32_t* out_a, int32_t* out_b, int64_t cap,
                            hipStream_t s) {
  const int64_t ub = n_ub < cap ? n_ub : cap;
  hipLaunchKernelGGL(k_pair_rows, dim3(grid_for(ub, 256, 4096)), dim3(256), 0, s, ids, n_ptr, pa, pb, sel, out_a,
                     out_b, cap);
  return hipGetLastError();
}

}  // namespace aiq
