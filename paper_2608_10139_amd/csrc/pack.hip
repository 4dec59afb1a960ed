// Packing of the selected rows into one variable-length token batch, and the
// device-side chunk descriptors that stand in for static shapes.
//
// The paper's prototype pads every row to a static maximum length and feeds
// fixed micro-batches through the model (Section 3.2 scan loop; Section 5
// names dynamic shapes as future work).  Here sequence i (the prompt prefix
// followed by selected row i's token list) occupies packed[cu[i] .. cu[i+1])
// with no padding, and the packed batch is cut at sequence boundaries into
// chunks of at most chunk_tokens + longest-sequence tokens.  Every count
// lives in device memory; kernels read their real extents from it.
#include "aiq_internal.h"
#include "dev_util.h"

namespace aiq {

static int grid_for(int64_t n, int threads, int cap = 4096) {
  int64_t g = (n + threads - 1) / threads;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return static_cast<int>(g);
}

__device__ __forceinline__ void set_status(int64_t* ctr, int64_t bits) {
  atomicOr(reinterpret_cast<unsigned long long*>(ctr + C_STATUS), static_cast<unsigned long long>(bits));
}


// ------------------------------------------------------------------ gather
// One wave per sequence: the prompt prefix, then the row's tokens.  Token ids
// outside [0, vocab) are flagged and replaced by 0 so later gathers stay in
// bounds.  The next sequence's extents are read while the current one is
// copied, and each lane keeps four token loads in flight.
__global__ __launch_bounds__(256) void k_gather(const int32_t* sel, const int64_t* n_ptr, const int64_t* off,
                                                const int32_t* tokens, const int64_t* cu, Prefix pre,
                                                int32_t vocab, int64_t t_ub, int32_t* packed, int64_t* ctr) {
  const int64_t n = *n_ptr;
  const int lane = threadIdx.x & 63;
  const int64_t wave = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6;
  const int64_t n_waves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  bool bad = false;
  // extents of sequence i: packed [c0, c1), source tokens + s0
  auto extents = [&](int64_t i, int64_t& c0, int64_t& c1, int64_t& s0) {
    c0 = cu[i];
    c1 = cu[i + 1];
    s0 = off[sel[i]];
  };
  int64_t i = wave;
  int64_t c0 = 0, c1 = 0, s0 = 0;
  if (i < n) extents(i, c0, c1, s0);
  while (i < n) {
    const int64_t in = i + n_waves;
    int64_t d0 = 0, d1 = 0, t0 = 0;
    if (in < n) extents(in, d0, d1, t0);   // in flight during the copy below
    if (c1 > t_ub) {   // more tokens than the table declared: never written
      bad = true;
    } else {
      int32_t* dst = packed + c0;
      for (int j = lane; j < pre.n; j += 64) dst[j] = pre.tok[j];
      const int64_t L = c1 - c0 - pre.n;
      const int32_t* src = tokens + s0;
      int32_t* out = dst + pre.n;
      int64_t j = lane;
      for (; j + 192 < L; j += 256) {
        int32_t v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = src[j + 64 * u];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          if (v[u] < 0 || v[u] >= vocab) {
            bad = true;
            v[u] = 0;
          }
          out[j + 64 * u] = v[u];
        }
      }
      for (; j < L; j += 64) {
        int32_t t = src[j];
        if (t < 0 || t >= vocab) {
          bad = true;
          t = 0;
        }
        out[j] = t;
      }
    }
    i = in;
    c0 = d0;
    c1 = d1;
    s0 = t0;
  }
  if (bad) set_status(ctr, AIQ_DEV_TOKEN_RANGE);
}

hipError_t launch_gather_tokens(const int32_t* sel, const int64_t* n_ptr, int64_t n_ub,
                                const int64_t* offsets, const int32_t* tokens, const int64_t* cu,
                                const Prefix& prefix, int32_t vocab, int64_t t_ub, int32_t* packed,
                                int64_t* ctr, hipStream_t s) {
  hipLaunchKernelGGL(k_gather, dim3(grid_for(n_ub, 4, 8192)), dim3(256), 0, s, sel, n_ptr, offsets,
                     tokens, cu, prefix, vocab, t_ub, packed, ctr);
  return hipGetLastError();
}

// ------------------------------------------------------------------ chunk descriptors
// Chunk c holds the sequences whose key cu[i] + i lies in
// [c*chunk_tokens, (c+1)*chunk_tokens): every sequence counts as one unit
// besides its tokens, so a chunk holds at most chunk_tokens sequences even
// when lists are empty.  The last chunk also takes any sequence beyond the
// bound (none when n_chunks * chunk_tokens exceeds tokens + sequences, which
// the plan guarantees).
__device__ __forceinline__ int64_t lower_bound_cu(const int64_t* cu, int64_t n, int64_t v) {
  int64_t lo = 0, hi = n;  // first i in [0, n) with key(i) >= v, else n
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    if (cu[mid] + mid < v) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

__global__ void k_chunk_desc(const int64_t* cu, const int64_t* n_ptr, int64_t chunk_tokens, int64_t n_chunks,
                             int64_t t_ub, int64_t* desc) {
  // only sequences that end inside the packed buffer take part
  int64_t n = *n_ptr;
  {
    int64_t lo = 0, hi = n;   // first i with cu[i + 1] > t_ub
    while (lo < hi) {
      const int64_t mid = (lo + hi) >> 1;
      if (cu[mid + 1] > t_ub) hi = mid;
      else lo = mid + 1;
    }
    n = lo;
  }
  for (int64_t c = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; c < n_chunks; c += (int64_t)gridDim.x * blockDim.x) {
    const int64_t sb = lower_bound_cu(cu, n, c * chunk_tokens);
    const int64_t se = c + 1 == n_chunks ? n : lower_bound_cu(cu, n, (c + 1) * chunk_tokens);
    int64_t* d = desc + c * D_STRIDE;
    d[D_TOK_BEGIN] = cu[sb];
    d[D_NTOK] = cu[se] - cu[sb];
    d[D_SEQ_BEGIN] = sb;
    d[D_NSEQ] = se - sb;
  }
}

hipError_t launch_chunk_desc(const int64_t* cu, const int64_t* n_ptr, int64_t chunk_tokens,
                             int64_t n_chunks, int64_t t_ub, int64_t* desc, hipStream_t s) {
  hipLaunchKernelGGL(k_chunk_desc, dim3(grid_for(n_chunks, 256)), dim3(256), 0, s, cu, n_ptr,
                     chunk_tokens, n_chunks, t_ub, desc);
  return hipGetLastError();
}

// prefill-only entry: one chunk covering a caller-packed batch.  One
// workgroup checks cu_seqlens (starts at 0, ends at n_tok, every sequence at
// least one token); a malformed array empties the chunk and sets a status bit
// so no later kernel indexes outside the caller's buffers.
__global__ __launch_bounds__(1024) void k_packed_desc(const int32_t* cu32, int32_t n_seq, int64_t n_tok,
                                                      int64_t* cu64, int64_t* desc, int64_t* ctr) {
  int bad = 0;
  for (int64_t i = threadIdx.x; i <= n_seq; i += blockDim.x) {
    const int64_t v = cu32[i];
    cu64[i] = v;
    if (i == 0 && v != 0) bad = 1;
    if (i == n_seq && v != n_tok) bad = 1;
    if (i < n_seq && static_cast<int64_t>(cu32[i + 1]) <= v) bad = 1;
  }
  bad = __syncthreads_or(bad);
  if (threadIdx.x == 0) {
    desc[D_TOK_BEGIN] = 0;
    desc[D_NTOK] = bad ? 0 : n_tok;
    desc[D_SEQ_BEGIN] = 0;
    desc[D_NSEQ] = bad ? 0 : n_seq;
    ctr[C_NSEQ] = bad ? 0 : n_seq;
    if (bad) ctr[C_STATUS] |= AIQ_DEV_LIST_LEN;
  }
}

hipError_t launch_packed_desc(const int32_t* cu32, int32_t n_seq, int64_t n_tok, int64_t* cu64,
                              int64_t* desc, int64_t* ctr, hipStream_t s) {
  hipLaunchKernelGGL(k_packed_desc, dim3(1), dim3(1024), 0, s, cu32, n_seq, n_tok, cu64, desc, ctr);
  return hipGetLastError();
}

// ------------------------------------------------------------------ shared prompt prefix
// The prefix alone as a packed batch of one sequence (its own prefill pass
// produces the keys and values every row attends to).
__global__ void k_prefix_batch(Prefix pre, int32_t* tok, int64_t* cu, int64_t* desc) {
  const int i = threadIdx.x;
  if (i < pre.n) tok[i] = pre.tok[i];
  if (i == 0) {
    cu[0] = 0;
    cu[1] = pre.n;
    desc[D_TOK_BEGIN] = 0;
    desc[D_NTOK] = pre.n;
    desc[D_SEQ_BEGIN] = 0;
    desc[D_NSEQ] = 1;
  }
}

hipError_t launch_prefix_batch(const Prefix& prefix, int32_t* tok, int64_t* cu, int64_t* desc, hipStream_t s) {
  if (prefix.n <= 0 || prefix.n > AIQ_MAX_PREFIX) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_prefix_batch, dim3(1), dim3(AIQ_MAX_PREFIX), 0, s, prefix, tok, cu, desc);
  return hipGetLastError();
}

__global__ void k_copy_row_f32(const float* src, float* dst, int32_t n) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) dst[i] = src[i];
}

hipError_t launch_copy_row_f32(const float* src, float* dst, int32_t n, hipStream_t s) {
  hipLaunchKernelGGL(k_copy_row_f32, dim3(1), dim3(256), 0, s, src, dst, n);
  return hipGetLastError();
}

// ------------------------------------------------------------------ rotary table
// cos / sin of pos * theta**(-2i/hd), evaluated in fp64 and rounded to fp32.
__global__ void k_rope_table(int32_t max_pos, int32_t half, double theta, int32_t hd, float* cos_t, float* sin_t,
                             float* rev) {
  const int64_t n = static_cast<int64_t>(max_pos) * half;
  if (blockIdx.x == 0 && static_cast<int>(threadIdx.x) < half) {
    const int i = threadIdx.x;
    rev[i] = static_cast<float>(pow(theta, -2.0 * static_cast<double>(i) / static_cast<double>(hd)) /
                                6.283185307179586);
  }
  for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < n; j += (int64_t)gridDim.x * blockDim.x) {
    const int64_t p = j / half;
    const int i = static_cast<int>(j % half);
    const double inv = pow(theta, -2.0 * static_cast<double>(i) / static_cast<double>(hd));
    const double a = static_cast<double>(p) * inv;
    cos_t[j] = static_cast<float>(cos(a));
    sin_t[j] = static_cast<float>(sin(a));
  }
}

hipError_t launch_rope_table(int32_t max_pos, int32_t half, double theta, int32_t hd, float* cos_t,
                             float* sin_t, float* rev, hipStream_t s) {
  hipLaunchKernelGGL(k_rope_table, dim3(grid_for(static_cast<int64_t>(max_pos) * half, 256)), dim3(256), 0,
                     s, max_pos, half, theta, hd, cos_t, sin_t, rev);
  return hipGetLastError();
}

// ------------------------------------------------------------------ embedding
// One wave per chunk token (grid-stride): x[t, :] = E[tok, :] in fp32 and
// pos[t] = position of the token inside its own sequence, found by a 64-way
// search of the chunk's sequence offsets (each round narrows the range 64x).
// With a norm gain `g` (MFMA path) the wave also writes h[t, :] = x * g in 16
// bits and rs[t] = 1 / sqrt(mean(x^2) + eps): the first RMSNorm, applied by
// the first projection.
__device__ __forceinline__ int64_t seq_of(const int64_t* cu, int64_t sb, int64_t ns, int64_t gt, int lane) {
  int64_t lo = sb, n = ns;   // answer in [lo, lo + n): the last i with cu[i] <= gt
  while (n > 1) {
    const int64_t step = (n + 63) / 64;
    const int64_t i = lo + lane * step;
    const bool le = i < lo + n && cu[i] <= gt;
    const uint64_t b = __ballot(le);
    if (b == 0) break;   // cannot happen (cu[lo] <= gt holds throughout); keeps the index in range
    const int last = 63 - __builtin_clzll(b);
    lo += static_cast<int64_t>(last) * step;
    const int64_t rem = n - static_cast<int64_t>(last) * step;
    n = rem < step ? rem : step;
  }
  return lo;
}

template <bool NORM>
__global__ __launch_bounds__(256) void k_embed(const int64_t* desc, const int64_t* cu, const int32_t* packed,
                                               const void* emb, int32_t wdtype, int32_t d, int32_t vocab,
                                               float* x, int32_t* pos, int64_t* ctr, const float* g, float eps,
                                               void* h, int32_t h_act, float* rs, int32_t pos_base) {
  const int64_t tb = desc[D_TOK_BEGIN], nt = desc[D_NTOK], sb = desc[D_SEQ_BEGIN], ns = desc[D_NSEQ];
  const int lane = threadIdx.x & 63;
  const int64_t wave = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6;
  const int64_t n_waves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t t = wave; t < nt; t += n_waves) {
    const int64_t gt = tb + t;
    int32_t tok = packed[gt];
    if (tok < 0 || tok >= vocab) {   // only reachable through caller-packed batches
      if (lane == 0) set_status(ctr, AIQ_DEV_TOKEN_RANGE);
      tok = 0;
    }
    const int64_t sq = seq_of(cu, sb, ns, gt, lane);
    if (lane == 0) pos[t] = pos_base + static_cast<int32_t>(gt - cu[sq]);
    float* xr = x ? x + t * d : nullptr;   // null: x is not written (the first projection reads the table)
    float ssq = 0.f;
    for (int c = lane * 4; c < d; c += 256) {
      float4 o;
      if (wdtype == AIQ_BF16 || wdtype == AIQ_F16) {
        const int ea = wdtype == AIQ_F16 ? ACT_F16 : ACT_BF16;
        const uint16_t* er = static_cast<const uint16_t*>(emb) + static_cast<int64_t>(tok) * d;
        const uint2 v = *reinterpret_cast<const uint2*>(er + c);
        o.x = act2f(static_cast<uint16_t>(v.x & 0xFFFFu), ea);
        o.y = act2f(static_cast<uint16_t>(v.x >> 16), ea);
        o.z = act2f(static_cast<uint16_t>(v.y & 0xFFFFu), ea);
        o.w = act2f(static_cast<uint16_t>(v.y >> 16), ea);
      } else {
        o = *reinterpret_cast<const float4*>(static_cast<const float*>(emb) + static_cast<int64_t>(tok) * d + c);
      }
      if (x) *reinterpret_cast<float4*>(xr + c) = o;
      if (NORM) {
        const float4 gv = *reinterpret_cast<const float4*>(g + c);
        uint2 hv;
        hv.x = f2act(o.x * gv.x, h_act) | (static_cast<uint32_t>(f2act(o.y * gv.y, h_act)) << 16);
        hv.y = f2act(o.z * gv.z, h_act) | (static_cast<uint32_t>(f2act(o.w * gv.w, h_act)) << 16);
        *reinterpret_cast<uint2*>(static_cast<uint16_t*>(h) + t * d + c) = hv;
        ssq += (o.x * o.x + o.y * o.y) + (o.z * o.z + o.w * o.w);
      }
    }
    if (NORM) {
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) ssq += __shfl_xor(ssq, o);
      if (lane == 0) rs[t] = 1.0f / sqrtf(ssq / static_cast<float>(d) + eps);
    }
  }
}

hipError_t launch_embed(const int64_t* desc, const int64_t* cu, const int32_t* packed,
                        const void* emb, int32_t wdtype, int32_t d, int32_t vocab, float* x, int32_t* pos,
                        int64_t* ctr, int64_t t_cap, hipStream_t s) {
  hipLaunchKernelGGL(k_embed<false>, dim3(grid_for(t_cap, 4, 8192)), dim3(256), 0, s, desc, cu, packed, emb,
                     wdtype, d, vocab, x, pos, ctr, nullptr, 0.f, nullptr, 0, nullptr, 0);
  return hipGetLastError();
}

hipError_t launch_embed_norm(const int64_t* desc, const int64_t* cu, const int32_t* packed, const void* emb,
                             int32_t wdtype, int32_t d, int32_t vocab, float* x, int32_t* pos, int64_t* ctr,
                             const float* g, float eps, void* h, int32_t h_act, float* rs, int64_t t_cap,
                             hipStream_t s, int32_t pos_base) {
  if (h_act == ACT_F32) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_embed<true>, dim3(grid_for(t_cap, 4, 8192)), dim3(256), 0, s, desc, cu, packed, emb,
                     wdtype, d, vocab, x, pos, ctr, g, eps, h, h_act, rs, pos_base);
  return hipGetLastError();
}

// ------------------------------------------------------------------ weight conversion
// bf16 -> fp16, element by element: the bf16 value widened exactly to fp32,
// then rounded to the nearest fp16 (ties to even; values below 2^-14 become
// fp16 subnormals, above 65504 infinities), 8 elements per thread in 16-byte
// pieces plus a scalar tail.
__global__ void k_bf16_to_f16(const uint16_t* src, uint16_t* dst, int64_t n) {
  const int64_t n8 = n / 8;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n8; i += stride) {
    const uint4 v = reinterpret_cast<const uint4*>(src)[i];
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    uint32_t o[4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
      o[k] = f2h(bf2f(static_cast<uint16_t>(w[k] & 0xFFFFu))) |
             (static_cast<uint32_t>(f2h(bf2f(static_cast<uint16_t>(w[k] >> 16)))) << 16);
    reinterpret_cast<uint4*>(dst)[i] = make_uint4(o[0], o[1], o[2], o[3]);
  }
  for (int64_t i = n8 * 8 + blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += stride)
    dst[i] = f2h(bf2f(src[i]));
}

hipError_t launch_bf16_to_f16(const void* src, void* dst, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_bf16_to_f16, dim3(grid_for(n / 8 + 1, 256, 8192)), dim3(256), 0, s,
                     static_cast<const uint16_t*>(src), static_cast<uint16_t*>(dst), n);
  return hipGetLastError();
}

}  // namespace aiq
