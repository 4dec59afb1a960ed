// AI_TRANSFORM: greedy generation after the prefill (Table 1 maps it to a
// causal-LM forward with generative decoding, output masked with a pad id;
// Section 4, Q3 and Q5), and the LIKE match over the generated tokens.
//
// A generation step runs one row per sequence of the chunk through the same
// projections as the prefill (M = number of sequences), a decode attention
// kernel over the sequence's kept keys and values, and the full-vocabulary
// head as a GEMM whose epilogue keeps only each row's maximum per 64 columns,
// followed by a row argmax over those.  Keys and values
// of the prompt stay where the prefill put them (the chunk's per-layer q|k|v
// rows, plus the shared prefix's rows); those of generated tokens go to a
// per-layer cache [sequence][step][2 d_kv].  Everything runs on the launch
// stream; counts come from device memory.
#include "aiq_internal.h"
#include "dev_util.h"

namespace aiq {

static int grid_for(int64_t n, int per_block, int cap) {
  int64_t g = (n + per_block - 1) / per_block;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return static_cast<int>(g);
}

__device__ __forceinline__ float wave_sum_g(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ float wave_max_g(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

// ------------------------------------------------------------------ descriptors
__global__ void k_gen_desc(const int64_t* cd, int64_t* gd, int64_t* cnt, int32_t nb) {
  const int64_t n = cd[D_NSEQ];
  if (threadIdx.x == 0) {
    gd[D_TOK_BEGIN] = 0;
    gd[D_NTOK] = n;
    gd[D_SEQ_BEGIN] = cd[D_SEQ_BEGIN];
    gd[D_NSEQ] = n;
  }
  for (int b = threadIdx.x; b < nb; b += blockDim.x) {
    const int64_t r = n - static_cast<int64_t>(b) * GEN_HEAD_ROWS;
    cnt[b] = r < 0 ? 0 : (r > GEN_HEAD_ROWS ? GEN_HEAD_ROWS : r);
  }
}

hipError_t launch_gen_desc(const int64_t* chunk_desc, int64_t* gen_desc, int64_t* cnt, int32_t n_blocks,
                           hipStream_t s) {
  hipLaunchKernelGGL(k_gen_desc, dim3(1), dim3(256), 0, s, chunk_desc, gen_desc, cnt, n_blocks);
  return hipGetLastError();
}

// ------------------------------------------------------------------ last positions of a chunk
// The label head needs only each sequence's last position, and in the last
// layer nothing after the q|k|v projection feeds any other position: that
// layer's attention (for the last query), O projection, norm and FFN run on
// one row per sequence, in blocks of R sequences.
__global__ void k_last_desc(const int64_t* cd, int64_t* ld, int32_t nb, int64_t R) {
  const int64_t n = cd[D_NSEQ];
  for (int b = threadIdx.x; b < nb; b += blockDim.x) {
    int64_t r = n - static_cast<int64_t>(b) * R;
    r = r < 0 ? 0 : (r > R ? R : r);
    int64_t* o = ld + static_cast<int64_t>(b) * D_STRIDE;
    o[D_TOK_BEGIN] = cd[D_TOK_BEGIN];
    o[D_NTOK] = r;
    o[D_SEQ_BEGIN] = cd[D_SEQ_BEGIN] + static_cast<int64_t>(b) * R;
    o[D_NSEQ] = r;
  }
}

hipError_t launch_last_desc(const int64_t* chunk_desc, int64_t* ldesc, int32_t nb, int64_t R, hipStream_t s) {
  if (nb <= 0 || R <= 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_last_desc, dim3(1), dim3(256), 0, s, chunk_desc, ldesc, nb, R);
  return hipGetLastError();
}

// Wave per sequence, 16-byte pieces of the row.
__global__ __launch_bounds__(256) void k_last_rows(const int64_t* ld, const int64_t* cu, const float* x, int32_t d,
                                                   float* xl) {
  const int64_t n = ld[D_NSEQ], sb = ld[D_SEQ_BEGIN], tb = ld[D_TOK_BEGIN];
  const int lane = threadIdx.x & 63;
  const int64_t wave = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6;
  const int64_t n_waves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t i = wave; i < n; i += n_waves) {
    const int64_t c1 = cu[sb + i + 1];
    if (c1 == cu[sb + i]) continue;
    const float4* src = reinterpret_cast<const float4*>(x + (c1 - 1 - tb) * d);
    float4* dst = reinterpret_cast<float4*>(xl + i * d);
    for (int c = lane; c < d / 4; c += 64) dst[c] = src[c];
  }
}

// Wave per sequence: the row of d 16-bit values in 16-byte pieces.
__global__ __launch_bounds__(256) void k_last_h(const int64_t* ld, const int64_t* cu, const uint16_t* h,
                                                const float* rs, const int32_t* pos, int32_t d, uint16_t* hl,
                                                float* rsl, int32_t* posl) {
  const int64_t n = ld[D_NSEQ], sb = ld[D_SEQ_BEGIN], tb = ld[D_TOK_BEGIN];
  const int lane = threadIdx.x & 63;
  const int64_t wave = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6;
  const int64_t n_waves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t i = wave; i < n; i += n_waves) {
    const int64_t c1 = cu[sb + i + 1];
    if (c1 == cu[sb + i]) continue;
    const int64_t r = c1 - 1 - tb;
    const uint4* src = reinterpret_cast<const uint4*>(h + r * d);
    uint4* dst = reinterpret_cast<uint4*>(hl + i * d);
    for (int c = lane; c < d / 8; c += 64) dst[c] = src[c];
    if (lane == 0) {
      rsl[i] = rs[r];
      posl[i] = pos[r];
    }
  }
}

hipError_t launch_last_h(const int64_t* ldesc, const int64_t* cu, const void* h, const float* rs, const int32_t* pos,
                         int32_t d, void* hl, float* rsl, int32_t* posl, int64_t R, hipStream_t s) {
  if (d % 8) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_last_h, dim3(grid_for(R, 4, 8192)), dim3(256), 0, s, ldesc, cu,
                     static_cast<const uint16_t*>(h), rs, pos, d, static_cast<uint16_t*>(hl), rsl, posl);
  return hipGetLastError();
}

hipError_t launch_last_rows(const int64_t* ldesc, const int64_t* cu, const float* x, int32_t d, float* xl,
                            int64_t R, hipStream_t s) {
  if (d % 4) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_last_rows, dim3(grid_for(R, 4, 8192)), dim3(256), 0, s, ldesc, cu, x, d, xl);
  return hipGetLastError();
}

// ------------------------------------------------------------------ embedding of the current tokens
// Wave per sequence: x = E[tok], h = x * g (16-bit), rs = 1 / rms(x), and the
// position after the prompt (shared prefix included) and the earlier steps.
__global__ __launch_bounds__(256) void k_gen_embed(const int64_t* gd, const int64_t* cu, const int32_t* tok,
                                                   int32_t step, int32_t npre, const uint16_t* emb, int32_t ea,
                                                   int32_t d, int32_t vocab, float* x, int32_t* pos, const float* g,
                                                   float eps, uint16_t* h, int32_t h_act, float* rs) {
  const int64_t n = gd[D_NSEQ], sb = gd[D_SEQ_BEGIN];
  const int lane = threadIdx.x & 63;
  const int64_t wave = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6;
  const int64_t n_waves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t i = wave; i < n; i += n_waves) {
    int32_t t = tok[i];
    if (t < 0 || t >= vocab) t = 0;   // argmax ids are in range; keeps the gather in bounds regardless
    if (lane == 0) pos[i] = npre + static_cast<int32_t>(cu[sb + i + 1] - cu[sb + i]) + step;
    const uint16_t* er = emb + static_cast<int64_t>(t) * d;
    float* xr = x + i * d;
    float ssq = 0.f;
    for (int c = lane * 4; c < d; c += 256) {
      const uint2 v = *reinterpret_cast<const uint2*>(er + c);
      float4 o;
      o.x = act2f(static_cast<uint16_t>(v.x & 0xFFFFu), ea);
      o.y = act2f(static_cast<uint16_t>(v.x >> 16), ea);
      o.z = act2f(static_cast<uint16_t>(v.y & 0xFFFFu), ea);
      o.w = act2f(static_cast<uint16_t>(v.y >> 16), ea);
      *reinterpret_cast<float4*>(xr + c) = o;
      const float4 gv = *reinterpret_cast<const float4*>(g + c);
      uint2 hv;
      hv.x = f2act(o.x * gv.x, h_act) | (static_cast<uint32_t>(f2act(o.y * gv.y, h_act)) << 16);
      hv.y = f2act(o.z * gv.z, h_act) | (static_cast<uint32_t>(f2act(o.w * gv.w, h_act)) << 16);
      *reinterpret_cast<uint2*>(h + i * d + c) = hv;
      ssq += (o.x * o.x + o.y * o.y) + (o.z * o.z + o.w * o.w);
    }
    ssq = wave_sum_g(ssq);
    if (lane == 0) rs[i] = 1.0f / sqrtf(ssq / static_cast<float>(d) + eps);
  }
}

hipError_t launch_gen_embed(const int64_t* gen_desc, const int64_t* cu, const int32_t* tok, int32_t step,
                            int32_t npre, const void* emb, int32_t wdtype, int32_t d, int32_t vocab, float* x,
                            int32_t* pos, const float* g, float eps, void* h, int32_t h_act, float* rs,
                            int64_t seq_ub, hipStream_t s) {
  if ((wdtype != AIQ_BF16 && wdtype != AIQ_F16) || h_act == ACT_F32 || d % 4) return hipErrorInvalidValue;
  const int ea = wdtype == AIQ_F16 ? ACT_F16 : ACT_BF16;
  hipLaunchKernelGGL(k_gen_embed, dim3(grid_for(seq_ub, 4, 8192)), dim3(256), 0, s, gen_desc, cu, tok, step, npre,
                     static_cast<const uint16_t*>(emb), ea, d, vocab, x, pos, g, eps, static_cast<uint16_t*>(h),
                     h_act, rs);
  return hipGetLastError();
}

// ------------------------------------------------------------------ decode attention
// Wave per (sequence, K/V head): the REP = n_heads / n_kv query heads of the
// group against every kept key of the sequence (prompt, earlier generated
// tokens, this token).  A key row of HD fp16 values is read by LPK = HD / 8
// lanes, 16 bytes each, so one wave load covers 64 / LPK whole rows; keys go
// in blocks of 4 such loads (an online-softmax step), the next block's key
// and value rows in flight while the current one is used.  Each lane keeps
// its 8 query dims and 8 output dims per head; partial dot products meet
// over the LPK lanes of a row, partial outputs over the key groups at the
// end.  The wave also stores this step's key and value into the generated
// cache.
template <int HD, int REP>
__global__ __launch_bounds__(256) void k_attn_gen(GenAttnArgs a) {
  constexpr int LPK = HD / 8;     // lanes per key row
  constexpr int KPI = 64 / LPK;   // key rows per wave load
  constexpr int IT = 4;           // wave loads per block
  constexpr int KB = KPI * IT;    // keys per online-softmax block
  const int64_t n = a.gen_desc[D_NSEQ], sb = a.gen_desc[D_SEQ_BEGIN], tb = a.chunk_desc[D_TOK_BEGIN];
  const int lane = threadIdx.x & 63, gk = lane / LPK, c = lane % LPK;
  const int64_t wave = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6;
  const int64_t n_waves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  const int d_q = a.n_heads * HD, d_kv = a.n_kv * HD;
  const float scale = 1.4426950408889634f / sqrtf(static_cast<float>(HD));   // log2(e) / sqrt(hd)
  const uint16_t* qkv = static_cast<const uint16_t*>(a.qkv);
  const uint16_t* kvc = static_cast<const uint16_t*>(a.kvc);
  const uint16_t* pkv = static_cast<const uint16_t*>(a.pkv);
  uint16_t* gkv = static_cast<uint16_t*>(a.gkv);
  uint16_t* out = static_cast<uint16_t*>(a.out);
  const int64_t ld = a.ld;
  const int64_t items = n * a.n_kv;

  for (int64_t item = wave; item < items; item += n_waves) {
    const int64_t i = item / a.n_kv;
    const int kvh = static_cast<int>(item % a.n_kv);
    const int64_t s0 = a.cu[sb + i] - tb;
    const int own = static_cast<int>(a.cu[sb + i + 1] - a.cu[sb + i]);
    const int P = a.npre + own;   // prompt positions
    if (a.last_row && own == 0) continue;   // no own row to attend from (same for the whole wave)
    // keys: the prompt, the earlier generated tokens, this token (last-row
    // mode: the prompt, whose last row is the query)
    const int N = a.last_row ? P : P + a.step + 1;
    const uint16_t* qrow = !a.last_row ? qkv + i * ld : (qkv ? qkv + i * a.ldq : kvc + (s0 + own - 1) * ld);
    const int kc = d_q + kvh * HD, vc = d_q + d_kv + kvh * HD;   // key / value columns of a q|k|v row
    uint16_t* gslot = a.last_row ? nullptr : gkv + (i * a.gen + a.step) * (2 * d_kv);
    if (!a.last_row && lane < 2 * LPK) {
      const bool isv = lane >= LPK;
      const int cc = lane % LPK;
      *reinterpret_cast<uint4*>(gslot + (isv ? d_kv : 0) + kvh * HD + cc * 8) =
          *reinterpret_cast<const uint4*>(qrow + (isv ? vc : kc) + cc * 8);
    }
    float qf[REP][8];
#pragma unroll
    for (int r = 0; r < REP; ++r) {
      const uint4 u = *reinterpret_cast<const uint4*>(qrow + (kvh * REP + r) * HD + c * 8);
      const uint32_t uw[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        qf[r][2 * e] = h2f(static_cast<uint16_t>(uw[e] & 0xFFFFu)) * scale;
        qf[r][2 * e + 1] = h2f(static_cast<uint16_t>(uw[e] >> 16)) * scale;
      }
    }
    // this lane's 16-byte pieces of key j's key and value rows
    auto rows_of = [&](int j, const uint16_t*& kp, const uint16_t*& vp) {
      const uint16_t* row;
      int ko = kc, vo = vc;
      if (j < a.npre) {
        row = pkv + static_cast<int64_t>(j) * ld;
      } else if (j < P) {
        row = kvc + (s0 + j - a.npre) * ld;
      } else if (j < P + a.step) {
        row = gkv + (i * a.gen + (j - P)) * (2 * d_kv);
        ko = kvh * HD;
        vo = d_kv + kvh * HD;
      } else {
        row = qrow;
      }
      kp = row + ko + c * 8;
      vp = row + vo + c * 8;
    };
    auto load_block = [&](int kb, uint4 (&kr)[IT], uint4 (&vr)[IT]) {
#pragma unroll
      for (int it = 0; it < IT; ++it) {
        const int j = kb + it * KPI + gk;
        kr[it] = make_uint4(0, 0, 0, 0);
        vr[it] = make_uint4(0, 0, 0, 0);
        if (j < N) {
          const uint16_t *kp, *vp;
          rows_of(j, kp, vp);
          kr[it] = *reinterpret_cast<const uint4*>(kp);
          vr[it] = *reinterpret_cast<const uint4*>(vp);
        }
      }
    };

    float m[REP], l[REP], o[REP][8];
#pragma unroll
    for (int r = 0; r < REP; ++r) {
      m[r] = -INFINITY;
      l[r] = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) o[r][e] = 0.f;
    }
    uint4 kr[IT], vr[IT];
    load_block(0, kr, vr);
    for (int kb = 0; kb < N; kb += KB) {
      uint4 kn[IT], vn[IT];
      if (kb + KB < N) load_block(kb + KB, kn, vn);   // next block in flight
      float s[REP][IT];
#pragma unroll
      for (int it = 0; it < IT; ++it) {
        const uint32_t uw[4] = {kr[it].x, kr[it].y, kr[it].z, kr[it].w};
        float kf[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          kf[2 * e] = h2f(static_cast<uint16_t>(uw[e] & 0xFFFFu));
          kf[2 * e + 1] = h2f(static_cast<uint16_t>(uw[e] >> 16));
        }
        const bool ok = kb + it * KPI + gk < N;
#pragma unroll
        for (int r = 0; r < REP; ++r) {
          float dot = 0.f;
#pragma unroll
          for (int e = 0; e < 8; ++e) dot = fmaf(qf[r][e], kf[e], dot);
#pragma unroll
          for (int off = 1; off < LPK; off <<= 1) dot += __shfl_xor(dot, off);
          s[r][it] = ok ? dot : -INFINITY;
        }
      }
      float vf[IT][8];
#pragma unroll
      for (int it = 0; it < IT; ++it) {
        const uint32_t uw[4] = {vr[it].x, vr[it].y, vr[it].z, vr[it].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          vf[it][2 * e] = h2f(static_cast<uint16_t>(uw[e] & 0xFFFFu));
          vf[it][2 * e + 1] = h2f(static_cast<uint16_t>(uw[e] >> 16));
        }
      }
#pragma unroll
      for (int r = 0; r < REP; ++r) {
        float mx = s[r][0];
#pragma unroll
        for (int it = 1; it < IT; ++it) mx = fmaxf(mx, s[r][it]);
        const float m_new = fmaxf(m[r], wave_max_g(mx));   // finite: key kb is valid
        const float alpha = exp2f(m[r] - m_new);
        float p[IT], ps = 0.f;
#pragma unroll
        for (int it = 0; it < IT; ++it) {
          p[it] = exp2f(s[r][it] - m_new);   // 0 for keys past the end (score -inf)
          ps += p[it];
        }
        // every key's probability sits in its LPK lanes: count it once
        l[r] = l[r] * alpha + wave_sum_g(c == 0 ? ps : 0.f);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          float acc = o[r][e] * alpha;
#pragma unroll
          for (int it = 0; it < IT; ++it) acc = fmaf(p[it], vf[it][e], acc);
          o[r][e] = acc;
        }
        m[r] = m_new;
      }
      if (kb + KB < N) {
#pragma unroll
        for (int it = 0; it < IT; ++it) {
          kr[it] = kn[it];
          vr[it] = vn[it];
        }
      }
    }
    // partial outputs of the key groups (lanes with the same dims) add up
#pragma unroll
    for (int r = 0; r < REP; ++r) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
#pragma unroll
        for (int off = LPK; off < 64; off <<= 1) o[r][e] += __shfl_xor(o[r][e], off);
      if (gk == 0) {
        const float inv = 1.0f / l[r];
        uint32_t pk[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
          pk[e] = f2act(o[r][2 * e] * inv, a.out_act) |
                  (static_cast<uint32_t>(f2act(o[r][2 * e + 1] * inv, a.out_act)) << 16);
        *reinterpret_cast<uint4*>(out + i * d_q + (kvh * REP + r) * HD + c * 8) = make_uint4(pk[0], pk[1], pk[2], pk[3]);
      }
    }
  }
}

hipError_t launch_attention_gen(const GenAttnArgs& a, hipStream_t s) {
  if (a.n_kv <= 0 || a.n_heads % a.n_kv || a.npre < 0 || (a.npre > 0 && !a.pkv) || a.out_act == ACT_F32 ||
      (!a.last_row && (a.step < 0 || a.step >= a.gen || !a.gkv || !a.qkv)))
    return hipErrorInvalidValue;
  const int rep = a.n_heads / a.n_kv;
  const dim3 grid(grid_for(a.seq_ub * a.n_kv, 4, 8192)), block(256);
#define AIQ_GEN_ATTN(HD_)                                                          \
  switch (rep) {                                                                   \
    case 1: hipLaunchKernelGGL((k_attn_gen<HD_, 1>), grid, block, 0, s, a); break; \
    case 2: hipLaunchKernelGGL((k_attn_gen<HD_, 2>), grid, block, 0, s, a); break; \
    case 3: hipLaunchKernelGGL((k_attn_gen<HD_, 3>), grid, block, 0, s, a); break; \
    case 4: hipLaunchKernelGGL((k_attn_gen<HD_, 4>), grid, block, 0, s, a); break; \
    case 8: hipLaunchKernelGGL((k_attn_gen<HD_, 8>), grid, block, 0, s, a); break; \
    default: return hipErrorInvalidValue;                                          \
  }
  if (a.hd == 64) {
    AIQ_GEN_ATTN(64)
  } else if (a.hd == 128) {
    AIQ_GEN_ATTN(128)
  } else {
    return hipErrorInvalidValue;
  }
#undef AIQ_GEN_ATTN
  return hipGetLastError();
}

// ------------------------------------------------------------------ final norm of the step rows
__global__ __launch_bounds__(256) void k_norm_rows(const int64_t* gd, const float* x, const float* g, int32_t d,
                                                   float eps, uint16_t* hf, int32_t act) {
  const int64_t n = gd[D_NSEQ];
  const int lane = threadIdx.x & 63;
  const int64_t wave = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6;
  const int64_t n_waves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t i = wave; i < n; i += n_waves) {
    const float* xr = x + i * d;
    float ss = 0.f;
    for (int c = lane; c < d; c += 64) ss += xr[c] * xr[c];
    ss = wave_sum_g(ss);
    const float r = 1.0f / sqrtf(ss / static_cast<float>(d) + eps);
    for (int c = lane; c < d; c += 64) hf[i * d + c] = f2act(xr[c] * r * g[c], act);
  }
}

hipError_t launch_norm_rows(const int64_t* gen_desc, const float* x, const float* g, int32_t d, float eps, void* hf,
                            int32_t act, int64_t seq_ub, hipStream_t s) {
  if (act == ACT_F32) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_norm_rows, dim3(grid_for(seq_ub, 4, 4096)), dim3(256), 0, s, gen_desc, x, g, d, eps,
                     static_cast<uint16_t*>(hf), act);
  return hipGetLastError();
}

// ------------------------------------------------------------------ argmax of the next token
// The head GEMM leaves, per row, the maximum and its column over every 64
// columns (lowest column on ties); a wave per row picks the largest, again
// the lowest column among equals, and records the token.
__global__ __launch_bounds__(256) void k_gen_argmax(const int2* part, int32_t n_chunk, const int64_t* cnt,
                                                    int64_t row0, const int64_t* gd, int32_t step, int32_t G,
                                                    int32_t eos, int32_t pad, int32_t* tok, int32_t* done,
                                                    int32_t* gen) {
  const int64_t rows = *cnt, sb = gd[D_SEQ_BEGIN];
  const int lane = threadIdx.x & 63;
  const int64_t wave = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6;
  const int64_t n_waves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t r = wave; r < rows; r += n_waves) {
    const int2* pr = part + r * n_chunk;
    float best = -INFINITY;
    int32_t bi = INT32_MAX;
    for (int c = lane; c < n_chunk; c += 64) {   // ascending columns: strict > keeps each lane's first maximum
      const int2 p = pr[c];
      const float v = __int_as_float(p.x);
      if (v > best) {
        best = v;
        bi = p.y;
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ov = __shfl_xor(best, o);
      const int32_t oi = __shfl_xor(bi, o);
      if (ov > best || (ov == best && oi < bi)) {
        best = ov;
        bi = oi;
      }
    }
    if (bi == INT32_MAX) bi = 0;   // no finite maximum (every logit NaN or -inf)
    if (lane == 0) {
      const int64_t i = row0 + r;
      const bool ended = done[i] != 0;
      gen[(sb + i) * G + step] = ended ? pad : bi;
      tok[i] = bi;
      if (!ended && bi == eos) done[i] = 1;
    }
  }
}

hipError_t launch_gen_argmax(const void* part, int32_t vocab, const int64_t* cnt, int64_t row0,
                             const int64_t* gen_desc, int32_t step, int32_t G, int32_t eos, int32_t pad,
                             int32_t* tok, int32_t* done, int32_t* gen, hipStream_t s) {
  if (vocab % 64) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_gen_argmax, dim3(grid_for(GEN_HEAD_ROWS, 4, 1024)), dim3(256), 0, s,
                     static_cast<const int2*>(part), vocab / 64, cnt, row0, gen_desc, step, G, eos, pad, tok, done,
                     gen);
  return hipGetLastError();
}

// ------------------------------------------------------------------ LIKE over the generated tokens
// Wave per selected row: the generated length (through the first end token),
// then every start position tested by one lane.
__global__ __launch_bounds__(256) void k_gen_like(const int32_t* gen, const int64_t* n_ptr, int32_t G, int32_t eos,
                                                  LikePattern pat, int32_t* label) {
  const int64_t n = *n_ptr;
  const int lane = threadIdx.x & 63;
  const int64_t wave = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6;
  const int64_t n_waves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t i = wave; i < n; i += n_waves) {
    const int32_t* gr = gen + i * G;
    int glen = G;
    if (eos >= 0) {
      for (int c = 0; c < G; c += 64) {
        const uint64_t b = __ballot(c + lane < G && gr[c + lane] == eos);
        if (b) {
          glen = c + __builtin_ctzll(b) + 1;
          break;
        }
      }
    }
    bool hit = false;
    if (pat.n == 0) {
      hit = true;
    } else {
      for (int s = lane; s + pat.n <= glen; s += 64) {
        bool ok = true;
        for (int q = 0; q < pat.n && ok; ++q) ok = gr[s + q] == pat.tok[q];
        hit = hit || ok;
      }
      hit = __ballot(hit) != 0;
    }
    if (lane == 0) label[i] = hit ? 1 : 0;
  }
}

hipError_t launch_gen_like(const int32_t* gen, const int64_t* n_ptr, int64_t n_ub, int32_t G, int32_t eos,
                           const LikePattern& pat, int32_t* label, hipStream_t s) {
  if (pat.n < 0 || pat.n > AIQ_MAX_LIKE || G <= 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_gen_like, dim3(grid_for(n_ub, 4, 4096)), dim3(256), 0, s, gen, n_ptr, G, eos, pat, label);
  return hipGetLastError();
}

__global__ void k_copy_rows_i32(const int32_t* src, const int64_t* n_ptr, int32_t per_row, int32_t* dst,
                                int64_t cap_rows) {
  int64_t rows = *n_ptr;
  if (rows > cap_rows) rows = cap_rows;
  const int64_t total = rows * per_row;
  for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < total; j += (int64_t)gridDim.x * blockDim.x)
    dst[j] = src[j];
}

hipError_t launch_copy_rows_i32(const int32_t* src, const int64_t* n_ptr, int64_t n_ub, int32_t per_row,
                                int32_t* dst, int64_t cap_rows, hipStream_t s) {
  const int64_t ub = (n_ub < cap_rows ? n_ub : cap_rows) * per_row;
  hipLaunchKernelGGL(k_copy_rows_i32, dim3(grid_for(ub, 256, 4096)), dim3(256), 0, s, src, n_ptr, per_row, dst,
                     cap_rows);
  return hipGetLastError();
}

}  // namespace aiq
