// Causal self-attention over the packed variable-length batch, grouped K/V
// heads (query head j reads K/V head j / (n_heads / n_kv)).
//
// Work items are (sequence, K/V head, head group) walked by a persistent
// grid; a workgroup holds REP of the n_heads / n_kv query heads that read one
// K/V head (all of them when registers allow), four waves per query head, so
// each staged key block serves all of them (its global reads happen once per
// group instead of once per query head).  An item loops over 64-query blocks of its own sequence and, inside,
// over 64-key blocks from the sequence start up to the diagonal, the next key
// block's global reads in flight while the current one is consumed.  Key
// blocks are aligned to the sequence start, so a row's result does not depend
// on the other rows packed next to it.  Softmax is the usual online form in fp32
// (running max and sum, rescaled output accumulator).
//
// MFMA path for bf16 models (hd 64 / 128): q, k, v arrive in fp16 and both
// products run on v_mfma_f32_16x16x32_f16 (fp16 keeps 3 more mantissa bits
// than bf16 at the same rate).  S^T = K Q^T puts one query per lane column and
// 4 keys per lane, which is exactly the operand layout the P V product needs
// for P^T, so probabilities never leave registers; V is staged row-major in
// LDS and read transposed by gfx950's ds_read_b64_tr_b16.  The softmax denominator sums the fp16-rounded probabilities that the
// P V product actually uses.
//
// Shared prompt prefix (MFMA path): a sequence is then the prefix's npre
// rows (pkv, computed once) followed by its own rows, with blocks and
// positions counted from the prefix start exactly as for the concatenated
// sequence; only the own rows are queries.  Each own query therefore meets
// the same key blocks, in the same order, as in the concatenated sequence.
#include "aiq_internal.h"
#include "dev_util.h"

#include <type_traits>

namespace aiq {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
typedef __attribute__((address_space(3))) uint16_t lds_u16;

// 16-byte chunk `ch` of LDS row r (see k_attn_bf16)
__device__ __forceinline__ int kswz(int r, int ch) { return ch ^ ((r >> 1) & 7); }
__device__ __forceinline__ int vswz(int r, int ch) { return ch ^ (r & 7); }

static int grid_cap(int64_t items, int cap) {
  int64_t g = items;
  if (g > cap) g = cap;
  if (g < 1) g = 1;
  return static_cast<int>(g);
}


// ======================================================================= bf16 MFMA
template <int HD, int REP>
__global__ __launch_bounds__(256 * REP) void k_attn_bf16(AttnArgs a) {
  constexpr int KB = 64;            // keys per block
  constexpr int CH = HD / 8;        // 16-byte chunks per K row
  constexpr int NT = 256 * REP;     // threads: four waves per query head of the group
  constexpr int PER = (KB * CH + NT - 1) / NT;   // chunks of K (and of V) per thread per block (at most)
  // K and V of one key block, row-major, 16-byte chunks XOR-swizzled by row
  // bits (K: rows 2i and 2i+1 share a pattern, so the 16 rows of a fragment
  // read hit distinct banks; V: the rows of a transposed read do)
  __shared__ __attribute__((aligned(16))) uint16_t Ks[KB * HD];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[KB * HD];

  lds_u16* const vs_lds = (lds_u16*)(Vs);   // LDS address space, for the transposing reads
  const int64_t tb = a.desc[D_TOK_BEGIN], sb = a.desc[D_SEQ_BEGIN], ns = a.desc[D_NSEQ];
  const int groups = a.n_heads / (a.n_kv * REP);   // head groups per K/V head
  const int64_t n_items = ns * a.n_kv * groups;
  const int t = threadIdx.x, lane = t & 63, g = lane >> 4, c16 = lane & 15;
  const int w = (t >> 6) & 3;      // the wave's 16 queries of a 64-query block
  const int hq = t >> 8;           // its query head inside the workgroup's group
  const int rep = a.n_heads / a.n_kv;
  const int d_q = a.n_heads * HD, d_kv = a.n_kv * HD;
  const int np = a.npre;
  const float scale = 1.4426950408889634f / sqrtf(static_cast<float>(HD));   // log2(e) / sqrt(hd)
  const uint16_t* qkv = static_cast<const uint16_t*>(a.qkv);
  const uint16_t* pkv = static_cast<const uint16_t*>(a.pkv);
  uint16_t* out = static_cast<uint16_t*>(a.out);

  // A task is one 64-query block of one (sequence, head) item.  The first
  // key block and the queries of the next task are read while the last key
  // block of the current one is consumed.
  struct Task {
    int64_t item, s0;   // item, first packed row of the sequence's own rows
    int L, qb, h0;       // positions (prefix + own), query block, first query head of the group
  };
  // first task of the first item at or after `item` that has own rows
  auto item_task = [&](int64_t item, Task& tk) -> bool {
    for (; item < n_items; item += gridDim.x) {
      const int per_seq = a.n_kv * groups;
      const int64_t si = static_cast<int32_t>(item) / per_seq;   // items < 2^31 (checked at launch)
      const int64_t c0 = a.cu[sb + si], c1 = a.cu[sb + si + 1];
      if (c1 > c0) {
        const int r = static_cast<int>(item - si * per_seq);   // K/V head r / groups, group r % groups
        tk.item = item;
        tk.s0 = c0 - tb;
        tk.L = static_cast<int>(c1 - c0) + np;
        tk.qb = np / KB;
        tk.h0 = r * REP;   // K/V head r / groups owns query heads (r / groups) * rep ..
        return true;
      }
    }
    return false;
  };
  auto advance = [&](const Task& c, Task& n) -> bool {
    if ((c.qb + 1) * KB < c.L) {
      n = c;
      n.qb = c.qb + 1;
      return true;
    }
    return item_task(c.item + gridDim.x, n);
  };
  // row of position p: the prefix's rows, then the sequence's own rows
  auto row_of = [&](const Task& tk, int p) {
    return p < np ? pkv + static_cast<int64_t>(p) * a.ld : qkv + (tk.s0 + p - np) * a.ld;
  };
  // this thread's K and V chunks of key block kb (zeros past L)
  uint4 kr[PER], vr[PER];
  auto fetch = [&](const Task& tk, int kb) {
    const int kvh = tk.h0 / rep;
    const int kcol = d_q + kvh * HD, vcol = d_q + d_kv + kvh * HD;
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int id = t + u * NT, r = id / CH, ch = id % CH;
      const int kk = kb * KB + r;
      kr[u] = make_uint4(0, 0, 0, 0);
      vr[u] = make_uint4(0, 0, 0, 0);
      if (id < KB * CH && kk < tk.L) {
        const uint16_t* row = row_of(tk, kk);
        kr[u] = *reinterpret_cast<const uint4*>(row + kcol + ch * 8);
        vr[u] = *reinterpret_cast<const uint4*>(row + vcol + ch * 8);
      }
    }
  };
  // this lane's query (column of S^T): 8 dims per 32-dim chunk, zeros unless own
  auto load_q = [&](const Task& tk, half8 (&qf)[HD / 32]) {
    const int qi = tk.qb * KB + w * 16 + c16;
    const bool own = qi >= np && qi < tk.L;
    const int h = tk.h0 + hq;
#pragma unroll
    for (int kc = 0; kc < HD / 32; ++kc) {
      if (own)
        qf[kc] = *reinterpret_cast<const half8*>(qkv + (tk.s0 + qi - np) * a.ld + h * HD + kc * 32 + g * 8);
      else
        qf[kc] = half8{};
    }
  };

  Task cur;
  if (!item_task(blockIdx.x, cur)) return;
  half8 qf[HD / 32];
  load_q(cur, qf);
  fetch(cur, 0);
  half8 ones;
#pragma unroll
  for (int i = 0; i < 8; ++i) ones[i] = static_cast<_Float16>(1.0f);

  for (;;) {
    const int qb = cur.qb, L = cur.L;
    const int qi = qb * KB + w * 16 + c16;
    f32x4 o[HD / 16];
#pragma unroll
    for (int db = 0; db < HD / 16; ++db) o[db] = f32x4{0.f, 0.f, 0.f, 0.f};
    // softmax denominator: the P V product against a block of ones, so it
    // sums exactly the fp16 probabilities the numerator uses
    f32x4 ol = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY;   // running maximum of the scaled scores
    Task nxt;
    bool has_next = false;
    half8 qn[HD / 32];

    for (int kb = 0; kb <= qb; ++kb) {
      __syncthreads();   // previous key block fully consumed
#pragma unroll
      for (int u = 0; u < PER; ++u) {
        const int id = t + u * NT, r = id / CH, ch = id % CH;
        if (id < KB * CH) {
          *reinterpret_cast<uint4*>(Ks + r * HD + (kswz(r, ch) << 3)) = kr[u];
          *reinterpret_cast<uint4*>(Vs + r * HD + (vswz(r, ch) << 3)) = vr[u];
        }
      }
      __syncthreads();
      if (kb < qb) {
        fetch(cur, kb + 1);
      } else {
        has_next = advance(cur, nxt);
        if (has_next) {
          fetch(nxt, 0);
          load_q(nxt, qn);
        }
      }

      // S^T block j: keys 16j.., lane holds keys 16j + 4g + e for query c16
      f32x4 sacc[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        sacc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
        const int krow = j * 16 + c16;
#pragma unroll
        for (int kc = 0; kc < HD / 32; ++kc) {
          const half8 kf = *reinterpret_cast<const half8*>(Ks + krow * HD + (kswz(krow, kc * 4 + g) << 3));
          sacc[j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(kf, qf[kc], sacc[j], 0, 0, 0);
        }
      }
      // Only the diagonal block has keys after some query or past the end
      // (every key of an earlier block precedes every query of this one).
      if (kb == qb) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int key = kb * KB + j * 16 + 4 * g + e;
            if (!(key <= qi && key < L)) sacc[j][e] = -INFINITY;
          }
      }
      float mx = sacc[0][0];
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) mx = fmaxf(mx, sacc[j][e]);
      // across the four 16-lane rows: v_permlane16_swap with both operands
      // the same value leaves rows (x0, x0, x2, x2) in one result and
      // (x1, x1, x3, x3) in the other; v_permlane32_swap then pairs the two
      // halves of the wave.  Plain VALU ops, not LDS round trips (2 % faster
      // than two lane shuffles through the LDS crossbar).
      {
        const auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
        mx = fmaxf(__uint_as_float(r16[0]), __uint_as_float(r16[1]));
        const auto r32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
        mx = fmaxf(__uint_as_float(r32[0]), __uint_as_float(r32[1]));
      }
      // scale > 0, so the maximum of the scaled scores is the scaled maximum;
      // it is finite: each block holds a key at or before every query
      const float m_new = fmaxf(m_run, mx * scale);
      // v_exp_f32: results below 2^-126 flush to zero, far below the fp16
      // probabilities they feed
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);   // 0 on the first block
      m_run = m_new;
      half8 pb[2];   // fp16 probabilities of keys 32u + {4g + e, 16 + 4g + e}
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        f32x8 pf;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          pf[e] = __builtin_amdgcn_exp2f(fmaf(sacc[2 * u][e], scale, -m_new));
          pf[4 + e] = __builtin_amdgcn_exp2f(fmaf(sacc[2 * u + 1][e], scale, -m_new));
        }
        pb[u] = __builtin_convertvector(pf, half8);
      }
#pragma unroll
      for (int db = 0; db < HD / 16; ++db) o[db] *= alpha;
      ol *= alpha;

      // O^T += V^T P^T over two 32-key halves.  V^T fragments come from the
      // row-major V block through transposing LDS reads: in each 16-lane
      // group, lane 4a + b receives element b of the 8-byte pieces addressed
      // by lanes a, a + 4, a + 8, a + 12.  Lane i of group g therefore
      // addresses key row 32u + 16h + 4g + i/4 at dims 16db + 4(i%4), and lane
      // c16 receives dim 16db + c16 of those four keys: the keys its pb half h
      // holds.
#pragma unroll
      for (int u = 0; u < 2; ++u) {
#pragma unroll
        for (int db = 0; db < HD / 16; ++db) {
          v4i16 part[2];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int vrow = 32 * u + 16 * h + 4 * g + (c16 >> 2);
            const int dim = db * 16 + 4 * (c16 & 3);
            const int el = vrow * HD + (vswz(vrow, dim >> 3) << 3) + (dim & 7);
            part[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(reinterpret_cast<lds_v4i16*>(vs_lds + el));
          }
          const half8 vf = __builtin_bit_cast(half8, __builtin_shufflevector(part[0], part[1], 0, 1, 2, 3, 4, 5, 6, 7));
          o[db] = __builtin_amdgcn_mfma_f32_16x16x32_f16(vf, pb[u], o[db], 0, 0, 0);
        }
        ol = __builtin_amdgcn_mfma_f32_16x16x32_f16(ones, pb[u], ol, 0, 0, 0);
      }
    }
    if (qi >= np && qi < L) {
      const float inv = 1.0f / ol[0];
      uint16_t* orow = out + (cur.s0 + qi - np) * a.ldo + (cur.h0 + hq) * HD;
      // output type chosen once, not per element
      auto store = [&](auto f16_tag) {
        constexpr bool F16 = decltype(f16_tag)::value;
        auto cv = [](float f) { return F16 ? f2h(f) : f2bf(f); };
#pragma unroll
        for (int db = 0; db < HD / 16; ++db) {
          const f32x4 v = o[db];
          uint2 pk;
          pk.x = cv(v[0] * inv) | (static_cast<uint32_t>(cv(v[1] * inv)) << 16);
          pk.y = cv(v[2] * inv) | (static_cast<uint32_t>(cv(v[3] * inv)) << 16);
          *reinterpret_cast<uint2*>(orow + db * 16 + 4 * g) = pk;
        }
      };
      if (a.out_act == ACT_F16)
        store(std::true_type{});
      else
        store(std::false_type{});
    }
    if (!has_next) break;
    cur = nxt;
#pragma unroll
    for (int kc = 0; kc < HD / 32; ++kc) qf[kc] = qn[kc];
  }
}

hipError_t launch_attention_bf16(const AttnArgs& a, hipStream_t s) {
  if (a.npre < 0 || (a.npre > 0 && !a.pkv)) return hipErrorInvalidValue;
  if (a.n_kv <= 0 || a.n_heads % a.n_kv) return hipErrorInvalidValue;
  const int rep = a.n_heads / a.n_kv;
  // query heads per workgroup: the largest divisor of rep up to 4 (64-dim
  // heads, 125 registers at 16 waves) or 3 (128-dim heads, 166 registers at 12)
  const int cap = a.hd == 128 ? 3 : 4;
  int hpw = 1;
  for (int d = 1; d <= cap; ++d)
    if (rep % d == 0) hpw = d;
  const int64_t items = a.seq_ub * a.n_kv * (rep / hpw);
  if (items >= (int64_t(1) << 31)) return hipErrorInvalidValue;   // 32-bit item numbers
  // about 32 query heads' worth of workgroups per CU: with work items of very
  // unequal length (sequence lengths spread 16..512) a fine grid balances the
  // tail better
  const int g = grid_cap(items, 8192 / hpw);
#define AIQ_ATTN(HD, R) hipLaunchKernelGGL((k_attn_bf16<HD, R>), dim3(g), dim3(256 * R), 0, s, a)
  if (a.hd == 64) {
    switch (hpw) {
      case 1: AIQ_ATTN(64, 1); break;
      case 2: AIQ_ATTN(64, 2); break;
      case 3: AIQ_ATTN(64, 3); break;
      default: AIQ_ATTN(64, 4); break;
    }
  } else if (a.hd == 128) {
    switch (hpw) {
      case 1: AIQ_ATTN(128, 1); break;
      case 2: AIQ_ATTN(128, 2); break;
      default: AIQ_ATTN(128, 3); break;
    }
  } else {
    return hipErrorInvalidValue;
  }
#undef AIQ_ATTN
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
