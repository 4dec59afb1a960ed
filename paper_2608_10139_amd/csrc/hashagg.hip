// GROUP BY over arbitrary int32 keys, and the join's build table staged for
// probing from LDS.
//
// GROUP BY (Table 1: SELECT ... GROUP BY as a masked segmented reduction;
// the group-by workload of Section 4 aggregates AVG(label), COUNT(*) per
// movie):
//   accumulate : each workgroup aggregates a range of the selected rows into
//                a private open-addressing table in LDS (key word, count, sum),
//                then merges its occupied slots into one table in global
//                memory with 64-bit atomics.  Counts and sums are integers,
//                so the result does not depend on the order of the atomics.
//   compact    : the occupied global slots become a dense list of
//                (order key, slot) pairs.
//   sort       : least-significant-digit radix sort of that list, four 8-bit
//                digits of the order key (the key with its sign bit flipped,
//                so unsigned order is signed order); each pass is a per-block
//                digit histogram, one scan over (digit, block) and a stable
//                scatter.
//   emit       : groups in ascending key order with COUNT, SUM and AVG =
//                SUM / COUNT in fp64.
// Every int32 value is a valid key (INT32_MIN included): a slot word is the
// key's 32 bits with bit 32 set, and 0 marks an empty slot.
//
// Join staging: the build side's hash table (built by linear probing in
// global memory) is rehashed by one workgroup into a table of 2^k slots,
// 2^k >= 2 x its entries, small enough for LDS; the one-launch compaction then
// copies it into each block's LDS and probes there.
#include "aiq_internal.h"

namespace aiq {

__device__ __forceinline__ uint64_t key_word(int32_t key) {
  return static_cast<uint64_t>(static_cast<uint32_t>(key)) | (1ull << 32);
}
__device__ __forceinline__ uint32_t mix32(uint32_t k) { return k * 0x9E3779B1u; }

__device__ __forceinline__ void flag(int64_t* ctr, int64_t bits) {
  atomicOr(reinterpret_cast<unsigned long long*>(ctr + C_STATUS), static_cast<unsigned long long>(bits));
}

__device__ __forceinline__ int64_t key_value(const void* p, int dt, int64_t i) {
  switch (dt) {
    case AIQ_I8: return static_cast<const int8_t*>(p)[i];
    case AIQ_I16: return static_cast<const int16_t*>(p)[i];
    default: return static_cast<const int32_t*>(p)[i];
  }
}

// ------------------------------------------------------------------ accumulate

constexpr int HA_THREADS = 256;
constexpr int HA_LDS_SLOTS = 2048;                 // private table per workgroup
constexpr int HA_ITEMS = HA_THREADS;               // rows per round, one per thread
constexpr int HA_FLUSH_AT = HA_LDS_SLOTS / 2 - HA_ITEMS;   // occupancy that triggers a merge

// Adds (count, sum) to the global slot of key word kw.
__device__ __forceinline__ void global_add(const HashAggArgs& g, uint64_t kw, uint64_t c, uint64_t s,
                                           int64_t* ctr) {
  const uint32_t mask = (1u << g.cap_log2) - 1u;
  uint32_t h = mix32(static_cast<uint32_t>(kw)) >> (32 - g.cap_log2);
  for (uint32_t i = 0; i <= mask; ++i) {
    unsigned long long* w = reinterpret_cast<unsigned long long*>(g.slot + h);
    uint64_t cur = __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (cur == 0) cur = atomicCAS(w, 0ull, static_cast<unsigned long long>(kw));
    if (cur == 0 || cur == kw) {
      atomicAdd(reinterpret_cast<unsigned long long*>(g.cnt + h), static_cast<unsigned long long>(c));
      if (s) atomicAdd(reinterpret_cast<unsigned long long*>(g.sum + h), static_cast<unsigned long long>(s));
      return;
    }
    h = (h + 1) & mask;
  }
  flag(ctr, AIQ_DEV_HASH_FULL);
}

// mode 1: key = key_col[sel[i]], value = label[i], every selected row i.
// mode 2: key = payload[i], value 0, rows with label[i] == 1 only.
__global__ __launch_bounds__(HA_THREADS) void k_hagg_acc(const int32_t* sel, const int32_t* label,
                                                         const int32_t* payload, const int64_t* n_ptr,
                                                         const void* key_col, int32_t key_dt, int mode,
                                                         HashAggArgs g, int64_t* ctr) {
  __shared__ uint64_t lk[HA_LDS_SLOTS];
  __shared__ uint64_t ls[HA_LDS_SLOTS];
  __shared__ uint32_t lc[HA_LDS_SLOTS];
  __shared__ int used;
  const int t = threadIdx.x;
  const int64_t n = *n_ptr;
  auto clear = [&]() {
    for (int i = t; i < HA_LDS_SLOTS; i += HA_THREADS) {
      lk[i] = 0;
      ls[i] = 0;
      lc[i] = 0;
    }
    if (t == 0) used = 0;
  };
  auto merge = [&]() {
    for (int i = t; i < HA_LDS_SLOTS; i += HA_THREADS)
      if (lk[i]) global_add(g, lk[i], lc[i], ls[i], ctr);
  };
  clear();
  __syncthreads();
  const int64_t stride = static_cast<int64_t>(gridDim.x) * HA_ITEMS;
  for (int64_t i0 = static_cast<int64_t>(blockIdx.x) * HA_ITEMS; i0 < n; i0 += stride) {
    const int64_t i = i0 + t;
    bool take = i < n;
    int32_t key = 0;
    uint64_t val = 0;
    if (take) {
      if (mode == 1) {
        key = static_cast<int32_t>(key_value(key_col, key_dt, sel[i]));
        val = static_cast<uint64_t>(static_cast<int64_t>(label[i]));
      } else {
        take = label[i] == 1;
        key = payload[i];
      }
    }
    if (take) {
      const uint64_t kw = key_word(key);
      uint32_t h = mix32(static_cast<uint32_t>(key)) >> (32 - 11);   // log2(HA_LDS_SLOTS) = 11
      for (;;) {   // the table is never full (merged at half load), so a slot is found
        uint64_t cur = lk[h];
        if (cur == 0) {
          cur = atomicCAS(reinterpret_cast<unsigned long long*>(&lk[h]), 0ull, static_cast<unsigned long long>(kw));
          if (cur == 0) atomicAdd(&used, 1);
        }
        if (cur == 0 || cur == kw) {
          atomicAdd(&lc[h], 1u);
          if (val) atomicAdd(reinterpret_cast<unsigned long long*>(&ls[h]), static_cast<unsigned long long>(val));
          break;
        }
        h = (h + 1) & (HA_LDS_SLOTS - 1);
      }
    }
    __syncthreads();
    const int u = used;
    __syncthreads();   // every thread has read `used` before the next round changes it
    if (u > HA_FLUSH_AT) {   // the next round could push the load past one half
      merge();
      __syncthreads();
      clear();
      __syncthreads();
    }
  }
  merge();
}
static_assert(HA_LDS_SLOTS == 1 << 11, "LDS slot hash uses 11 bits");
static_assert(HA_FLUSH_AT > 0, "flush threshold");

// ------------------------------------------------------------------ compact
// Occupied slots -> (order key, slot), appended at positions reserved by one
// atomic per workgroup (the order is arbitrary; the sort fixes it).
constexpr int HC_THREADS = 256;
constexpr int HC_SLOTS = 16 * HC_THREADS;

__global__ __launch_bounds__(HC_THREADS) void k_hagg_compact(HashAggArgs g, uint32_t* okey, uint32_t* oslot,
                                                             int64_t* n_groups) {
  __shared__ int cnt;
  __shared__ int64_t base;
  const int t = threadIdx.x;
  const int64_t cap = int64_t(1) << g.cap_log2;
  const int64_t s0 = static_cast<int64_t>(blockIdx.x) * HC_SLOTS;
  if (t == 0) cnt = 0;
  __syncthreads();
  int mine = 0;
  for (int u = 0; u < HC_SLOTS / HC_THREADS; ++u) {
    const int64_t s = s0 + u * HC_THREADS + t;
    mine += (s < cap && g.slot[s] != 0) ? 1 : 0;
  }
  const int first = atomicAdd(&cnt, mine);
  __syncthreads();
  if (t == 0) base = cnt ? static_cast<int64_t>(atomicAdd(reinterpret_cast<unsigned long long*>(n_groups),
                                                          static_cast<unsigned long long>(cnt)))
                         : 0;
  __syncthreads();
  int64_t p = base + first;
  for (int u = 0; u < HC_SLOTS / HC_THREADS; ++u) {
    const int64_t s = s0 + u * HC_THREADS + t;
    if (s < cap) {
      const uint64_t kw = g.slot[s];
      if (kw) {
        okey[p] = static_cast<uint32_t>(kw) ^ 0x80000000u;
        oslot[p] = static_cast<uint32_t>(s);
        ++p;
      }
    }
  }
}

// ------------------------------------------------------------------ radix sort
// Items per block RS_ITEMS; histogram layout hist[digit * nblk + block] so
// that one exclusive scan gives every (digit, block) its first output slot.
constexpr int RS_THREADS = 256;
constexpr int RS_ROUNDS = 16;
constexpr int RS_ITEMS = RS_THREADS * RS_ROUNDS;

__global__ __launch_bounds__(RS_THREADS) void k_rs_hist(const uint32_t* key, const int64_t* n_ptr, int shift,
                                                        int64_t nblk, int64_t* hist) {
  __shared__ int h[256];
  const int t = threadIdx.x;
  const int64_t n = *n_ptr;
  const int64_t b = blockIdx.x;
  h[t] = 0;
  __syncthreads();
  for (int r = 0; r < RS_ROUNDS; ++r) {
    const int64_t i = b * RS_ITEMS + r * RS_THREADS + t;
    if (i < n) atomicAdd(&h[(key[i] >> shift) & 255u], 1);
  }
  __syncthreads();
  hist[static_cast<int64_t>(t) * nblk + b] = h[t];
}

// In-place exclusive scan of n int64 values by one workgroup of 1024 threads.
__global__ __launch_bounds__(1024) void k_scan_inplace(int64_t* v, int64_t n) {
  __shared__ int64_t ws[16];
  constexpr int PER = 16;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  int64_t carry = 0;
  for (int64_t b0 = 0; b0 < n; b0 += 1024 * PER) {
    const int64_t first = b0 + static_cast<int64_t>(t) * PER;
    int64_t x[PER];
    int64_t sum = 0;
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      x[k] = first + k < n ? v[first + k] : 0;
      sum += x[k];
    }
    int64_t incl = sum;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int64_t y = __shfl_up(incl, o);
      if (lane >= o) incl += y;
    }
    if (lane == 63) ws[w] = incl;
    __syncthreads();
    int64_t before = 0, all = 0;
    for (int i = 0; i < 16; ++i) {
      if (i < w) before += ws[i];
      all += ws[i];
    }
    __syncthreads();
    int64_t run = carry + before + incl - sum;
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      if (first + k < n) v[first + k] = run;
      run += x[k];
    }
    carry += all;
  }
}

// Stable scatter: round r takes items r * 256 + t of the block, so item order
// is (round, thread).  Inside a wave, lanes with the same digit find each
// other with eight ballots; earlier waves of the round and earlier rounds are
// counted in LDS.
__global__ __launch_bounds__(RS_THREADS) void k_rs_scatter(const uint32_t* key, const uint32_t* val,
                                                           const int64_t* n_ptr, int shift, int64_t nblk,
                                                           const int64_t* hist, uint32_t* okey, uint32_t* oval) {
  constexpr int W = RS_THREADS / 64;
  __shared__ int64_t base[256];
  __shared__ int wc[W][256];
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int64_t n = *n_ptr;
  const int64_t b = blockIdx.x;
  if (b * RS_ITEMS >= n) return;
  base[t] = hist[static_cast<int64_t>(t) * nblk + b];
#pragma unroll
  for (int k = 0; k < W; ++k) wc[k][t] = 0;
  __syncthreads();
  const uint64_t lt = lane ? (~0ull >> (64 - lane)) : 0ull;
  for (int r = 0; r < RS_ROUNDS; ++r) {
    const int64_t i = b * RS_ITEMS + r * RS_THREADS + t;
    const bool ok = i < n;
    uint32_t k = 0, v = 0, d = 0;
    if (ok) {
      k = key[i];
      v = val[i];
      d = (k >> shift) & 255u;
    }
    uint64_t peers = __ballot(ok);
#pragma unroll
    for (int bit = 0; bit < 8; ++bit) {
      const uint64_t set = __ballot((d >> bit) & 1u);
      peers &= ((d >> bit) & 1u) ? set : ~set;
    }
    const int rank = __popcll(peers & lt);
    if (ok && rank == 0) wc[w][d] = __popcll(peers);
    __syncthreads();
    if (ok) {
      int64_t pos = base[d] + rank;
      for (int q = 0; q < w; ++q) pos += wc[q][d];
      okey[pos] = k;
      oval[pos] = v;
    }
    __syncthreads();
    int add = 0;
#pragma unroll
    for (int q = 0; q < W; ++q) {
      add += wc[q][t];
      wc[q][t] = 0;
    }
    base[t] += add;
    __syncthreads();
  }
}

// ------------------------------------------------------------------ emit
__global__ void k_hagg_emit(const uint32_t* key, const uint32_t* slot, const int64_t* n_groups, HashAggArgs g,
                            int mode, int32_t* key_out, int64_t* cnt_out, int64_t* sum_out, double* avg_out,
                            int64_t cap, int64_t* ctr) {
  const int64_t n = *n_groups;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n && i < cap;
       i += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t s = slot[i];
    const int64_t c = g.cnt[s];
    const int64_t sm = mode == 1 ? g.sum[s] : 0;
    key_out[i] = static_cast<int32_t>(key[i] ^ 0x80000000u);
    cnt_out[i] = c;
    sum_out[i] = sm;
    avg_out[i] = mode == 1 ? static_cast<double>(sm) / static_cast<double>(c) : 0.0;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    ctr[C_GROUPS] = n < cap ? n : cap;
    if (n > cap) flag(ctr, AIQ_DEV_GROUP_CAP);
  }
}

int64_t hash_group_sort_blocks(int64_t max_groups) { return (max_groups + RS_ITEMS - 1) / RS_ITEMS; }

hipError_t launch_hash_group(const int32_t* sel, const int32_t* label, const int32_t* payload, const int64_t* n_ptr,
                             int64_t n_ub, const void* key_col, int32_t key_dtype, int mode, HashAggArgs g,
                             int64_t max_groups, int32_t* key_out, int64_t* cnt_out, int64_t* sum_out,
                             double* avg_out, int64_t cap, int64_t* ctr, hipStream_t s) {
  if (g.cap_log2 < 6 || g.cap_log2 > 31 || (int64_t(1) << g.cap_log2) < 2 * max_groups) return hipErrorInvalidValue;
  const int64_t cap_slots = int64_t(1) << g.cap_log2;
  hipError_t e = launch_fill_i64(reinterpret_cast<int64_t*>(g.slot), 3 * cap_slots, 0, s);   // slot, cnt, sum
  if (e != hipSuccess) return e;
  e = launch_fill_i64(g.n_groups, 1, 0, s);
  if (e != hipSuccess) return e;
  int64_t blocks = (n_ub + HA_ITEMS - 1) / HA_ITEMS;
  if (blocks > 512) blocks = 512;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_hagg_acc, dim3(static_cast<unsigned>(blocks)), dim3(HA_THREADS), 0, s, sel, label, payload,
                     n_ptr, key_col, key_dtype, mode, g, ctr);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(k_hagg_compact, dim3(static_cast<unsigned>((cap_slots + HC_SLOTS - 1) / HC_SLOTS)),
                     dim3(HC_THREADS), 0, s, g, g.key0, g.val0, g.n_groups);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const int64_t nblk = hash_group_sort_blocks(max_groups);
  uint32_t *kin = g.key0, *vin = g.val0, *kout = g.key1, *vout = g.val1;
  for (int shift = 0; shift < 32; shift += 8) {
    hipLaunchKernelGGL(k_rs_hist, dim3(static_cast<unsigned>(nblk)), dim3(RS_THREADS), 0, s, kin, g.n_groups, shift,
                       nblk, g.hist);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_scan_inplace, dim3(1), dim3(1024), 0, s, g.hist, 256 * nblk);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_rs_scatter, dim3(static_cast<unsigned>(nblk)), dim3(RS_THREADS), 0, s, kin, vin,
                       g.n_groups, shift, nblk, g.hist, kout, vout);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    uint32_t* tk = kin;
    kin = kout;
    kout = tk;
    uint32_t* tv = vin;
    vin = vout;
    vout = tv;
  }
  // four passes: the sorted list is back in key0 / val0
  int64_t eb = (max_groups + 255) / 256;
  if (eb > 2048) eb = 2048;
  if (eb < 1) eb = 1;
  hipLaunchKernelGGL(k_hagg_emit, dim3(static_cast<unsigned>(eb)), dim3(256), 0, s, kin, vin, g.n_groups, g, mode,
                     key_out, cnt_out, sum_out, avg_out, cap, ctr);
  return hipGetLastError();
}

// ------------------------------------------------------------------ join staging
// One workgroup: counts the global table's entries and, when a table of
// 2^k >= 2 x entries slots (k >= 6) fits JOIN_LDS_SLOTS, rehashes them into
// it (in LDS, then copied out to st.keys / st.vals) and writes k to
// *st.log2_out; otherwise writes 0 (probes then use the global table).
__global__ __launch_bounds__(1024) void k_hash_stage(HashArgs h, StagedHash st) {
  __shared__ int32_t sk[JOIN_LDS_SLOTS];
  __shared__ int32_t sv[JOIN_LDS_SLOTS];
  __shared__ int total;
  const int t = threadIdx.x;
  const int64_t cap = int64_t(1) << h.cap_log2;
  if (t == 0) total = 0;
  __syncthreads();
  int mine = 0;
  for (int64_t s = t; s < cap; s += 1024) mine += h.keys[s] != HASH_EMPTY;
  atomicAdd(&total, mine);
  __syncthreads();
  int lg = 6;
  while (lg < 30 && (int64_t(1) << lg) < 2 * static_cast<int64_t>(total)) ++lg;
  if ((int64_t(1) << lg) > JOIN_LDS_SLOTS) {
    if (t == 0) *st.log2_out = 0;
    return;
  }
  const int m = 1 << lg;
  for (int i = t; i < m; i += 1024) sk[i] = HASH_EMPTY;
  __syncthreads();
  for (int64_t s = t; s < cap; s += 1024) {
    const int32_t key = h.keys[s];
    if (key == HASH_EMPTY) continue;
    const int32_t val = h.vals[s];
    uint32_t p = (static_cast<uint32_t>(key) * 0x9E3779B1u) >> (32 - lg);
    for (;;) {   // at most half full: a free slot exists
      const int32_t prev = atomicCAS(&sk[p], HASH_EMPTY, key);
      if (prev == HASH_EMPTY) {
        sv[p] = val;
        break;
      }
      p = (p + 1) & (m - 1);
    }
  }
  __syncthreads();
  for (int i = t; i < m; i += 1024) {
    st.keys[i] = sk[i];
    st.vals[i] = sv[i];
  }
  if (t == 0) *st.log2_out = lg;
}

hipError_t launch_hash_stage(HashArgs h, StagedHash st, hipStream_t s) {
  hipLaunchKernelGGL(k_hash_stage, dim3(1), dim3(1024), 0, s, h, st);
  return hipGetLastError();
}

}  // namespace aiq
