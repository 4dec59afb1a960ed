// RMSNorm of the residual stream, and the last-position label head.
//
// The semantic decision reads only the last position's logits of each row
// and only the label columns (Figure 2: logits[:, -1, :], then the Yes / No
// columns compared on chip).  The head therefore never forms the [tokens,
// vocab] logits: one wave per sequence normalises the last token's residual
// row in fp32 and takes K dot products with the label rows of the LM head.
#include "aiq_internal.h"
#include "dev_util.h"

namespace aiq {

static int grid_for(int64_t n, int per_block, int cap) {
  int64_t g = (n + per_block - 1) / per_block;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return static_cast<int>(g);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}


// ------------------------------------------------------------------ residual add + RMSNorm
// One wave per row.  With a pending projection output `delta` the residual
// stream is updated first (x += delta, fp32, written back), then
// out = x / sqrt(mean(x^2) + eps) * g.  The sum of squares is reduced in a
// fixed order inside the row, so a row's result does not depend on which
// other rows share the launch.
__global__ __launch_bounds__(256) void k_rmsnorm(const int64_t* desc, float* x, const float* delta, const float* g,
                                                 int32_t d, float eps, void* out, int32_t out_act) {
  const int64_t nt = desc[D_NTOK];
  const int lane = threadIdx.x & 63;
  const int64_t wave = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6;
  const int64_t n_waves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  const int nv = d >> 2;
  constexpr int MAXV = 16;   // d <= 64 lanes * 16 float4 = 4096
  for (int64_t t = wave; t < nt; t += n_waves) {
    float4* xr = reinterpret_cast<float4*>(x + t * d);
    float4 v[MAXV];
    float ss = 0.f;
#pragma unroll
    for (int j = 0; j < MAXV; ++j) {
      const int c = lane + 64 * j;
      if (c < nv) {
        float4 a = xr[c];
        if (delta) {
          const float4 b = reinterpret_cast<const float4*>(delta + t * d)[c];
          a.x += b.x; a.y += b.y; a.z += b.z; a.w += b.w;
          xr[c] = a;
        }
        v[j] = a;
        ss += a.x * a.x + a.y * a.y + a.z * a.z + a.w * a.w;
      }
    }
    ss = wave_sum(ss);
    const float r = 1.0f / sqrtf(ss / static_cast<float>(d) + eps);
    const float4* gr = reinterpret_cast<const float4*>(g);
#pragma unroll
    for (int j = 0; j < MAXV; ++j) {
      const int c = lane + 64 * j;
      if (c < nv) {
        const float4 a = v[j], w = gr[c];
        if (out_act != ACT_F32) {
          uint2 p;
          p.x = f2act(a.x * r * w.x, out_act) | (static_cast<uint32_t>(f2act(a.y * r * w.y, out_act)) << 16);
          p.y = f2act(a.z * r * w.z, out_act) | (static_cast<uint32_t>(f2act(a.w * r * w.w, out_act)) << 16);
          reinterpret_cast<uint2*>(static_cast<uint16_t*>(out) + t * d)[c] = p;
        } else {
          reinterpret_cast<float4*>(static_cast<float*>(out) + t * d)[c] =
              make_float4(a.x * r * w.x, a.y * r * w.y, a.z * r * w.z, a.w * r * w.w);
        }
      }
    }
  }
}

hipError_t launch_rmsnorm(const int64_t* desc, float* x, const float* delta, const float* g, int32_t d,
                          float eps, void* out, int32_t out_act, int64_t t_cap, hipStream_t s) {
  if (d > 64 * 4 * 16) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_rmsnorm, dim3(grid_for(t_cap, 4, 4096)), dim3(256), 0, s, desc, x, delta, g, d, eps, out,
                     out_act);
  return hipGetLastError();
}

// ------------------------------------------------------------------ row scale
// The RMSNorm scale of each token from the per-slice sums of squares that the
// residual projection wrote, added in slice order.  A block takes 128 tokens:
// their rows of sums come in with coalesced 16-byte loads into LDS (rows
// padded by one float: conflict-free), then one thread per token adds its row
// (rows wider than RS_MAX_PART: each thread reads its row directly).
constexpr int RS_TOK = 128, RS_MAX_PART = 64;

__global__ __launch_bounds__(256) void k_row_scale(const int64_t* desc, const float* ssp, int32_t n_part, int32_t d,
                                                   float eps, float* rs) {
  __shared__ float part[RS_TOK * (RS_MAX_PART + 1)];
  const int64_t nt = desc[D_NTOK];
  if (n_part > RS_MAX_PART || n_part % 4) {   // wide models: thread per token straight from memory
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < nt; t += (int64_t)gridDim.x * blockDim.x) {
      const float* p = ssp + t * n_part;
      float ss = 0.f;
      for (int k = 0; k < n_part; ++k) ss += p[k];
      rs[t] = 1.0f / sqrtf(ss / static_cast<float>(d) + eps);
    }
    return;
  }
  const int stride = n_part + 1;
  const int q4 = n_part / 4;   // 16-byte pieces per token
  for (int64_t t0 = static_cast<int64_t>(blockIdx.x) * RS_TOK; t0 < nt; t0 += static_cast<int64_t>(gridDim.x) * RS_TOK) {
    const int ntok = nt - t0 < RS_TOK ? static_cast<int>(nt - t0) : RS_TOK;
    const float4* src = reinterpret_cast<const float4*>(ssp + t0 * n_part);
    for (int e = threadIdx.x; e < ntok * q4; e += blockDim.x) {
      const float4 v = src[e];
      float* dst = part + (e / q4) * stride + (e % q4) * 4;
      dst[0] = v.x;
      dst[1] = v.y;
      dst[2] = v.z;
      dst[3] = v.w;
    }
    __syncthreads();
    if (threadIdx.x < ntok) {
      const float* p = part + threadIdx.x * stride;
      float ss = 0.f;
      for (int k = 0; k < n_part; ++k) ss += p[k];
      rs[t0 + threadIdx.x] = 1.0f / sqrtf(ss / static_cast<float>(d) + eps);
    }
    __syncthreads();
  }
}

hipError_t launch_row_scale(const int64_t* desc, const float* ssp, int32_t n_part, int32_t d, float eps,
                            float* rs, int64_t t_cap, hipStream_t s) {
  if (n_part <= 0) return hipErrorInvalidValue;
  const int per_block = (n_part > RS_MAX_PART || n_part % 4) ? 256 : RS_TOK;
  hipLaunchKernelGGL(k_row_scale, dim3(grid_for(t_cap, per_block, 4096)), dim3(256), 0, s, desc, ssp, n_part, d, eps,
                     rs);
  return hipGetLastError();
}

// ------------------------------------------------------------------ label head + decision
// Wave per sequence of the chunk.  label_out / logits_out are indexed by the
// global sequence number (seq_begin + local index).
__global__ __launch_bounds__(256) void k_head(HeadArgs a) {
  const int64_t tb = a.desc[D_TOK_BEGIN], sb = a.desc[D_SEQ_BEGIN], ns = a.desc[D_NSEQ];
  const int lane = threadIdx.x & 63;
  const int64_t wave = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6;
  const int64_t n_waves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  const int d = a.d;
  for (int64_t i = wave; i < ns; i += n_waves) {
    const int64_t gi = sb + i;
    // no own token: the shared prefix's last token, else every logit is 0
    const bool no_own = a.cu[gi + 1] == a.cu[gi];
    const bool empty = no_own && !a.x_pre;
    const bool pre = no_own && a.x_pre;
    const int64_t last = no_own ? 0 : (a.x_compact ? i : a.cu[gi + 1] - 1 - tb);
    const float* xr = pre ? a.x_pre : a.x + last * d;
    const float* dr = (a.delta && !pre) ? a.delta + last * d : nullptr;   // last layer's pending output
    // an empty sequence reads no row: its normalised state is 0
    auto xv = [&](int c) { return empty ? 0.f : dr ? xr[c] + dr[c] : xr[c]; };
    float ss = 0.f;
    for (int c = lane; c < d; c += 64) ss += xv(c) * xv(c);
    ss = wave_sum(ss);
    const float r = empty ? 0.f : 1.0f / sqrtf(ss / static_cast<float>(d) + a.eps);
    float lg[AIQ_MAX_LABELS];
    for (int k = 0; k < a.n_labels; ++k) {
      float acc = 0.f;
      if (a.wdtype == AIQ_BF16 || a.wdtype == AIQ_F16) {
        const int wa = a.wdtype == AIQ_F16 ? ACT_F16 : ACT_BF16;
        const uint16_t* w = static_cast<const uint16_t*>(a.lm_head) + static_cast<int64_t>(a.labels[k]) * d;
        for (int c = lane; c < d; c += 64) acc += (xv(c) * r * a.g[c]) * act2f(w[c], wa);
      } else {
        const float* w = static_cast<const float*>(a.lm_head) + static_cast<int64_t>(a.labels[k]) * d;
        for (int c = lane; c < d; c += 64) acc += (xv(c) * r * a.g[c]) * w[c];
      }
      lg[k] = wave_sum(acc);
    }
    if (a.hf_out) {
      if (a.hf_act != ACT_F32) {
        uint16_t* o = static_cast<uint16_t*>(a.hf_out) + i * d;
        for (int c = lane; c < d; c += 64) o[c] = f2act(xv(c) * r * a.g[c], a.hf_act);
      } else {
        float* o = static_cast<float*>(a.hf_out) + i * d;
        for (int c = lane; c < d; c += 64) o[c] = xv(c) * r * a.g[c];
      }
    }
    if (lane == 0) {
      if (a.logits_out)
        for (int k = 0; k < a.n_labels; ++k) a.logits_out[gi * a.n_labels + k] = lg[k];
      if (a.label_out) {
        int32_t lab;
        if (a.decision == AIQ_DECIDE_BINARY_GT) {
          lab = lg[0] > lg[1] ? 1 : 0;
        } else {
          int best = 0;
          for (int k = 1; k < a.n_labels; ++k)
            if (lg[k] > lg[best]) best = k;
          lab = a.labels[best];
        }
        a.label_out[gi] = lab;
      }
    }
  }
}

hipError_t launch_head(const HeadArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_head, dim3(grid_for(a.seq_ub, 4, 2048)), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace aiq
