// Causal self-attention over the packed variable-length batch, grouped K/V
// heads (query head j reads K/V head j / (n_heads / n_kv)).
//
// Work items are (sequence, query head) pairs walked by a persistent grid;
// each item loops over 64-query blocks of its own sequence and, inside, over
// 64-key blocks from the sequence start up to the diagonal, the next key
// block's global reads in flight while the current one is consumed.  Key blocks are
// aligned to the sequence start, so a row's result does not depend on the
// other rows packed next to it.  Softmax is the usual online form in fp32
// (running max and sum, rescaled output accumulator).
//
// MFMA path for bf16 models (hd 64 / 128): q, k, v arrive in fp16 and both
// products run on v_mfma_f32_16x16x32_f16 (fp16 keeps 3 more mantissa bits
// than bf16 at the same rate).  S^T = K Q^T puts one query per lane column and
// 4 keys per lane, which is exactly the operand layout the P V product needs
// for P^T, so probabilities never leave registers; V is staged transposed in
// LDS.  The softmax denominator sums the fp16-rounded probabilities that the
// P V product actually uses.
//
// Shared prompt prefix (MFMA path): a sequence is then the prefix's npre
// rows (pkv, computed once) followed by its own rows, with blocks and
// positions counted from the prefix start exactly as for the concatenated
// sequence; only the own rows are queries.  Each own query therefore meets
// the same key blocks, in the same order, as in the concatenated sequence.
#include "aiq_internal.h"
#include "dev_util.h"

namespace aiq {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

static int grid_cap(int64_t items, int cap) {
  int64_t g = items;
  if (g > cap) g = cap;
  if (g < 1) g = 1;
  return static_cast<int>(g);
}


// ======================================================================= bf16 MFMA
template <int HD>
__global__ __launch_bounds__(256) void k_attn_bf16(AttnArgs a) {
  constexpr int KB = 64;            // keys per block
  constexpr int CH = HD / 8;        // 16-byte chunks per K row
  __shared__ __attribute__((aligned(16))) uint16_t Ks[KB * HD];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[HD * KB];

  const int64_t tb = a.desc[D_TOK_BEGIN], sb = a.desc[D_SEQ_BEGIN], ns = a.desc[D_NSEQ];
  const int64_t n_items = ns * a.n_heads;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6, g = lane >> 4, c16 = lane & 15;
  const int rep = a.n_heads / a.n_kv;
  const int d_q = a.n_heads * HD, d_kv = a.n_kv * HD;
  const float scale = 1.4426950408889634f / sqrtf(static_cast<float>(HD));   // log2(e) / sqrt(hd)
  const uint16_t* qkv = static_cast<const uint16_t*>(a.qkv);
  const uint16_t* pkv = static_cast<const uint16_t*>(a.pkv);
  uint16_t* out = static_cast<uint16_t*>(a.out);

  for (int64_t item = blockIdx.x; item < n_items; item += gridDim.x) {
    const int64_t si = item / a.n_heads;
    const int h = static_cast<int>(item % a.n_heads);
    const int kvh = h / rep;
    const int64_t s0 = a.cu[sb + si] - tb;
    const int np = a.npre;
    const int Lo = static_cast<int>(a.cu[sb + si + 1] - a.cu[sb + si]);   // own rows
    if (Lo == 0) continue;
    const int L = Lo + np;   // positions 0 .. L-1, the first np in pkv
    const int qcol = h * HD, kcol = d_q + kvh * HD, vcol = d_q + d_kv + kvh * HD;
    // row of position p: the prefix's rows, then the sequence's own rows
    auto row_of = [&](int p) { return p < np ? pkv + static_cast<int64_t>(p) * a.ld : qkv + (s0 + p - np) * a.ld; };

    for (int qb = np / KB; qb * KB < L; ++qb) {
      const int qi = qb * KB + w * 16 + c16;   // this lane's query position (column of S^T)
      const bool q_own = qi >= np && qi < L;
      half8 qf[HD / 32];
#pragma unroll
      for (int kc = 0; kc < HD / 32; ++kc) {
        if (q_own)
          qf[kc] = *reinterpret_cast<const half8*>(qkv + (s0 + qi - np) * a.ld + qcol + kc * 32 + g * 8);
        else
          qf[kc] = half8{};
      }
      f32x4 o[HD / 16];
#pragma unroll
      for (int db = 0; db < HD / 16; ++db) o[db] = f32x4{0.f, 0.f, 0.f, 0.f};
      float m_run = -INFINITY, l_run = 0.f;

      // this thread's K and V chunks of a key block (zeros past L); the next
      // block's are read into registers while the current block is consumed
      constexpr int PER = KB * CH / 256;
      uint4 kr[PER], vr[PER];
      auto fetch = [&](int kb) {
#pragma unroll
        for (int u = 0; u < PER; ++u) {
          const int id = t + u * 256, r = id / CH, ch = id % CH;
          const int kk = kb * KB + r;
          kr[u] = make_uint4(0, 0, 0, 0);
          vr[u] = make_uint4(0, 0, 0, 0);
          if (kk < L) {
            const uint16_t* row = row_of(kk);
            kr[u] = *reinterpret_cast<const uint4*>(row + kcol + ch * 8);
            vr[u] = *reinterpret_cast<const uint4*>(row + vcol + ch * 8);
          }
        }
      };
      fetch(0);
      for (int kb = 0; kb <= qb; ++kb) {
        __syncthreads();   // previous key block fully consumed
#pragma unroll
        for (int u = 0; u < PER; ++u) {
          const int id = t + u * 256, r = id / CH, ch = id % CH;
          *reinterpret_cast<uint4*>(Ks + r * HD + ((ch ^ (r & 7)) << 3)) = kr[u];
          const uint32_t vw[4] = {vr[u].x, vr[u].y, vr[u].z, vr[u].w};
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int dim = ch * 8 + j;
            const uint16_t e = static_cast<uint16_t>(vw[j >> 1] >> ((j & 1) * 16));
            Vt[dim * KB + ((((r >> 2) ^ (dim & 15)) << 2) | (r & 3))] = e;
          }
        }
        __syncthreads();
        if (kb < qb) fetch(kb + 1);

        // S^T block j: keys 16j.., lane holds keys 16j + 4g + e for query c16
        f32x4 sacc[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          sacc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
          const int krow = j * 16 + c16;
#pragma unroll
          for (int kc = 0; kc < HD / 32; ++kc) {
            const half8 kf = *reinterpret_cast<const half8*>(Ks + krow * HD + (((kc * 4 + g) ^ (krow & 7)) << 3));
            sacc[j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(kf, qf[kc], sacc[j], 0, 0, 0);
          }
        }
        float mx = -INFINITY;
        float sv[16];
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int key = kb * KB + j * 16 + 4 * g + e;
            const bool valid = key <= qi && key < L;
            const float s = valid ? sacc[j][e] * scale : -INFINITY;
            sv[j * 4 + e] = s;
            mx = fmaxf(mx, s);
          }
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_new = fmaxf(m_run, mx);
        const float alpha = (m_new == -INFINITY) ? 1.f : exp2f(m_run - m_new);
        float psum = 0.f;
        uint16_t ph[16];   // fp16 probabilities fed to the P V product
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float pf = (m_new == -INFINITY || sv[i] == -INFINITY) ? 0.f : exp2f(sv[i] - m_new);
          ph[i] = f2h(pf);
          psum += h2f(ph[i]);
        }
        l_run = l_run * alpha + psum;
        m_run = m_new;
#pragma unroll
        for (int db = 0; db < HD / 16; ++db) o[db] *= alpha;

        // O^T += V^T P^T over two 32-key halves
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          half8 pb;
          {
            uint16_t tmp[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              tmp[e] = ph[(2 * u) * 4 + e];
              tmp[4 + e] = ph[(2 * u + 1) * 4 + e];
            }
            pb = *reinterpret_cast<const half8*>(tmp);
          }
#pragma unroll
          for (int db = 0; db < HD / 16; ++db) {
            const int dim = db * 16 + c16;
            const uint16_t* vrow = Vt + dim * KB;
            const uint2 lo = *reinterpret_cast<const uint2*>(vrow + (((8 * u + g) ^ (dim & 15)) << 2));
            const uint2 hi = *reinterpret_cast<const uint2*>(vrow + (((8 * u + 4 + g) ^ (dim & 15)) << 2));
            const uint4 vv = make_uint4(lo.x, lo.y, hi.x, hi.y);
            const half8 vf = *reinterpret_cast<const half8*>(&vv);
            o[db] = __builtin_amdgcn_mfma_f32_16x16x32_f16(vf, pb, o[db], 0, 0, 0);
          }
        }
      }
      float l_tot = l_run;
      l_tot += __shfl_xor(l_tot, 16);
      l_tot += __shfl_xor(l_tot, 32);
      if (q_own) {
        const float inv = 1.0f / l_tot;
        uint16_t* orow = out + (s0 + qi - np) * a.ldo + h * HD;
#pragma unroll
        for (int db = 0; db < HD / 16; ++db) {
          const f32x4 v = o[db];
          uint2 pk;
          pk.x = f2act(v[0] * inv, a.out_act) | (static_cast<uint32_t>(f2act(v[1] * inv, a.out_act)) << 16);
          pk.y = f2act(v[2] * inv, a.out_act) | (static_cast<uint32_t>(f2act(v[3] * inv, a.out_act)) << 16);
          *reinterpret_cast<uint2*>(orow + db * 16 + 4 * g) = pk;
        }
      }
    }
  }
}

hipError_t launch_attention_bf16(const AttnArgs& a, hipStream_t s) {
  if (a.npre < 0 || (a.npre > 0 && !a.pkv)) return hipErrorInvalidValue;
  const int g = grid_cap(a.seq_ub * a.n_heads, 4096);
  if (a.hd == 64)
    hipLaunchKernelGGL(k_attn_bf16<64>, dim3(g), dim3(256), 0, s, a);
  else if (a.hd == 128)
    hipLaunchKernelGGL(k_attn_bf16<128>, dim3(g), dim3(256), 0, s, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

// ======================================================================= fp32
// One wave per item; each lane owns one query of the 64-query block and walks
// the keys of the staged block in order with an online softmax.
template <int HD>
__global__ __launch_bounds__(64) void k_attn_f32(AttnArgs a) {
  __shared__ float Ks[64][HD];
  __shared__ float Vs[64][HD];
  const int64_t tb = a.desc[D_TOK_BEGIN], sb = a.desc[D_SEQ_BEGIN], ns = a.desc[D_NSEQ];
  const int64_t n_items = ns * a.n_heads;
  const int lane = threadIdx.x;
  const int rep = a.n_heads / a.n_kv;
  const int d_q = a.n_heads * HD, d_kv = a.n_kv * HD;
  const float scale = 1.0f / sqrtf(static_cast<float>(HD));
  const float* qkv = static_cast<const float*>(a.qkv);
  float* out = static_cast<float*>(a.out);
  for (int64_t item = blockIdx.x; item < n_items; item += gridDim.x) {
    const int64_t si = item / a.n_heads;
    const int h = static_cast<int>(item % a.n_heads);
    const int kvh = h / rep;
    const int64_t s0 = a.cu[sb + si] - tb;
    const int L = static_cast<int>(a.cu[sb + si + 1] - a.cu[sb + si]);
    for (int qb = 0; qb * 64 < L; ++qb) {
      const int qi = qb * 64 + lane;
      float q[HD], o[HD];
#pragma unroll
      for (int i = 0; i < HD; ++i) {
        q[i] = qi < L ? qkv[(s0 + qi) * a.ld + h * HD + i] : 0.f;
        o[i] = 0.f;
      }
      float m = -INFINITY, l = 0.f;
      for (int kb = 0; kb <= qb; ++kb) {
        __syncthreads();
        for (int id = lane; id < 64 * HD; id += 64) {
          const int r = id / HD, c = id % HD;
          const int kk = kb * 64 + r;
          const bool ok = kk < L;
          Ks[r][c] = ok ? qkv[(s0 + kk) * a.ld + d_q + kvh * HD + c] : 0.f;
          Vs[r][c] = ok ? qkv[(s0 + kk) * a.ld + d_q + d_kv + kvh * HD + c] : 0.f;
        }
        __syncthreads();
        for (int r = 0; r < 64; ++r) {
          const int key = kb * 64 + r;
          if (key > qi || key >= L) break;
          float s = 0.f;
#pragma unroll
          for (int i = 0; i < HD; ++i) s = fmaf(q[i], Ks[r][i], s);
          s *= scale;
          const float m_new = fmaxf(m, s);
          const float alpha = expf(m - m_new);
          const float pr = expf(s - m_new);
          l = l * alpha + pr;
#pragma unroll
          for (int i = 0; i < HD; ++i) o[i] = o[i] * alpha + pr * Vs[r][i];
          m = m_new;
        }
      }
      if (qi < L) {
        const float inv = 1.0f / l;
        float* orow = out + (s0 + qi) * a.ldo + h * HD;
#pragma unroll
        for (int i = 0; i < HD; ++i) orow[i] = o[i] * inv;
      }
    }
  }
}

hipError_t launch_attention_f32(const AttnArgs& a, hipStream_t s) {
  if (a.npre != 0) return hipErrorInvalidValue;   // no shared prefix on this path
  const int g = grid_cap(a.seq_ub * a.n_heads, 4096);
  switch (a.hd) {
    case 32: hipLaunchKernelGGL(k_attn_f32<32>, dim3(g), dim3(64), 0, s, a); break;
    case 64: hipLaunchKernelGGL(k_attn_f32<64>, dim3(g), dim3(64), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace aiq
