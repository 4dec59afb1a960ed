// Dense projections of the prefill: C[M, N] = A[M, K] . W[N, K]^T with fused
// epilogues (rotary embedding on q/k, SwiGLU, GELU, residual add).
//
// bf16 path (gfx950 MFMA): 256 x 256 output tile per 512-thread workgroup,
// K stepped by 64 through two LDS stages (2 x 64 KB) filled by 16-byte
// direct-to-LDS loads, the next stage in flight while the current one feeds
// the MFMAs.  Eight waves in a 2 x 4 grid each own a 128 x 64 sub-tile =
// 4 x 2 blocks of v_mfma_f32_32x32x16_bf16 (the 32x32 form sustains about
// twice the rate of the 16x16x32 form on gfx950).  The next tile's first
// stage is fetched while the epilogue of the current one runs.
//
// M (tokens in the chunk) is read from device memory; the grid is persistent
// (one workgroup per CU) and walks the tiles, so an empty chunk costs one
// launch and no work.
//
// fp32 path: a plain 64 x 64 LDS-tiled FMA kernel with the same row mapping
// and epilogues, used for fp32 models.
#include "aiq_internal.h"
#include "dev_util.h"

#include <type_traits>

namespace aiq {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

static int g_cus[64];

static int num_cus() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (g_cus[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    g_cus[dev] = n;
  }
  return g_cus[dev];
}


__device__ __forceinline__ uint2 pack_bf16x4(float a, float b, float c, float d) {
  uint2 p;
  p.x = f2bf(a) | (static_cast<uint32_t>(f2bf(b)) << 16);
  p.y = f2bf(c) | (static_cast<uint32_t>(f2bf(d)) << 16);
  return p;
}

__device__ __forceinline__ float silu(float g) { return g / (1.0f + expf(-g)); }
__device__ __forceinline__ float gelu_erf(float x) { return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f)); }

// Row of the q or k weight that produces GEMM column c of that section.
// For hd = 128 the two 64-column halves of a head are reordered so that one
// wave's 64 columns hold 32 complete rotary pairs (i, i + 64).
__device__ __forceinline__ int qk_row(int c, int hd) {
  const int head = c / hd, cc = c % hd;
  int dim = cc;
  if (hd == 128) {
    const int hh = cc >> 6, jj = cc & 63;
    dim = jj < 32 ? hh * 32 + jj : 64 + hh * 32 + (jj - 32);
  }
  return head * hd + dim;
}

template <int EPI, typename T>
__device__ __forceinline__ const T* b_row(const GemmArgs& a, int n) {
  if (EPI == EPI_QKV_ROPE) {
    // the bf16 kernel applies the rotary pairs in registers and needs the
    // reordered rows; the fp32 kernel keeps the natural order
    constexpr bool reorder = sizeof(T) == 2;
    if (n < a.n_q) return static_cast<const T*>(a.B0) + static_cast<int64_t>(reorder ? qk_row(n, a.hd) : n) * a.K;
    n -= a.n_q;
    if (n < a.n_kv) return static_cast<const T*>(a.B1) + static_cast<int64_t>(reorder ? qk_row(n, a.hd) : n) * a.K;
    n -= a.n_kv;
    return static_cast<const T*>(a.B2) + static_cast<int64_t>(n) * a.K;
  } else if (EPI == EPI_SWIGLU) {
    // interleave 32-row groups: gate rows 32b.., up rows 32b.., ... so each
    // 64-column wave slice holds 32 gate columns and the 32 matching up columns
    const int b32 = n >> 5, r = n & 31;
    const int row = (b32 >> 1) * 32 + r;
    return static_cast<const T*>((b32 & 1) ? a.B1 : a.B0) + static_cast<int64_t>(row) * a.K;
  } else {
    return static_cast<const T*>(a.B0) + static_cast<int64_t>(n) * a.K;
  }
}

// ======================================================================= 16-bit MFMA
// The MFMA path runs on bf16 or fp16 operands (H = fp16); both forms of
// v_mfma_f32_32x32x16 have the same rate.
template <bool H> struct Op16;
template <> struct Op16<false> {
  typedef bf16x8 V;
  static __device__ __forceinline__ f32x16_t mma(V a, V b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ uint16_t cvt(float f) { return f2bf(f); }
  static __device__ __forceinline__ float widen(uint16_t u) { return __uint_as_float(static_cast<uint32_t>(u) << 16); }
};
template <> struct Op16<true> {
  typedef half8 V;
  static __device__ __forceinline__ f32x16_t mma(V a, V b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ uint16_t cvt(float f) { return f2h(f); }
  static __device__ __forceinline__ float widen(uint16_t u) { return h2f(u); }
};
constexpr int GM = 256, GN = 256, GK = 64, GT = 512;

typedef f32x16_t f32x16;

// Accumulator layout (v_mfma_f32_32x32x16_bf16, activations as the first
// operand): acc[i][j][4g + e] holds C[m][n] with
//   m = m0 + wm*128 + i*32 + 8g + 4*(lane/32) + e,   n = n0 + wn*64 + j*32 + lane%32.
// A lane owns one column of each 32-wide block, so the rotary pair (j = 0
// lower half, j = 1 upper half of a head) and the SwiGLU pair (j = 0 gate,
// j = 1 up) sit in the same lane.
//
// q, k and v (attention operands) are stored in fp16: 10 mantissa bits where
// bf16 has 7, at the same MFMA rate; their magnitudes are O(1) after RMSNorm.
//
// Output goes through LDS: each wave owns an 8 KB slice of the idle LDS stage,
// writes a slab of its sub-tile there in row-major order, then stores whole
// 16-byte pieces of rows to global memory (8 store instructions per slab
// instead of one 2-byte store per value).

__device__ __forceinline__ float silu_fast(float g) {
  return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g));
}

// Writes a slab of `rows` x `cols` elements of type T from the wave's LDS slice
// (row-major, `cols` per row) to C[m][col_of(c)] for rows m < M, 16 B per lane.
template <typename T, typename ColMap>
__device__ __forceinline__ void flush_slab(const T* slab, int rows, int cols, T* C, int64_t ldc, int64_t m_first,
                                           int64_t M, int lane, ColMap col_of) {
  constexpr int PER = 16 / sizeof(T);               // elements per 16-byte piece
  const int pieces_per_row = cols / PER;
  const int total = rows * pieces_per_row;
  for (int p = lane; p < total; p += 64) {
    const int r = p / pieces_per_row, c = (p % pieces_per_row) * PER;
    const int64_t m = m_first + r;
    if (m < M)
      *reinterpret_cast<uint4*>(C + m * ldc + col_of(c)) = *reinterpret_cast<const uint4*>(slab + r * cols + c);
  }
}

// `rl` holds the tile's row scales (QKV, SwiGLU) or the following norm's gain
// for the tile's columns (residual), `pl` the tile's positions, both in LDS;
// `rev` the rotary frequencies of this lane's dims (revolutions per position)
// for the first and second 64-dim half of a head.  `prefetch` issues the next
// tile's first loads: the residual epilogue calls it after its first loads of
// x, so that those do not queue behind it; the others call it first.
template <int EPI, bool H, typename Prefetch>
__device__ __forceinline__ void epilogue_bf16(const GemmArgs& a, f32x16 (&acc)[4][2], int64_t m0, int n0,
                                              int64_t M, int wm, int wn, int lane, uint16_t* slice,
                                              const float* rl, const int32_t* pl, float2 rev, Prefetch prefetch) {
  const int l32 = lane & 31, hi = lane >> 5;
  const int nw = n0 + wn * 64;   // first GEMM column of this wave
  const int64_t mw = m0 + wm * 128;   // first row of this wave's sub-tile
  if (EPI == EPI_RESID || EPI == EPI_RESID_EMB) {
    // x += acc in place; with a following norm also h = x * g and, per row,
    // the sum of x^2 over this wave's 64 columns.  A slab of 32 rows x 64
    // columns goes through LDS; each lane then owns 4 columns of 8 rows, and
    // the 16 lanes of a row add their squares in a fixed butterfly order.  A
    // row's x for the next slab is read as soon as its slot is free, so those
    // reads are in flight while the rest of the slab is processed.
    float* slab = reinterpret_cast<float*>(slice);
    const int cg = (lane & 15) * 4;
    const bool norm = a.gnext != nullptr;
    uint16_t* hout = static_cast<uint16_t*>(a.hout);
    const int part = nw >> 6;
    auto row_of = [&](int i, int k) { return mw + i * 32 + (lane >> 4) + 4 * k; };
    // the residual before this projection: x, or (first layer) the token's
    // embedding row widened from 16 bits, which is exactly what x would hold
    const int64_t tok0 = EPI == EPI_RESID_EMB ? a.x_tok_desc[D_TOK_BEGIN] : 0;
    auto load_x = [&](int i, float4 (&v)[8]) {
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        int64_t m = row_of(i, k);
        if (m > M - 1) m = M - 1;   // in bounds; the value is not used
        if (EPI == EPI_RESID_EMB) {
          int32_t tok = a.x_tok[tok0 + m];
          if (tok < 0 || tok >= a.vocab) tok = 0;
          const uint2 e = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(a.x_emb) +
                                                          static_cast<int64_t>(tok) * a.ldc + nw + cg);
          v[k] = make_float4(Op16<H>::widen(static_cast<uint16_t>(e.x & 0xFFFFu)),
                             Op16<H>::widen(static_cast<uint16_t>(e.x >> 16)),
                             Op16<H>::widen(static_cast<uint16_t>(e.y & 0xFFFFu)),
                             Op16<H>::widen(static_cast<uint16_t>(e.y >> 16)));
        } else {
          v[k] = *reinterpret_cast<const float4*>(a.x + m * a.ldc + nw + cg);
        }
      }
    };
    float4 xo[8];
    load_x(0, xo);
    prefetch();
    float4 gv = make_float4(0.f, 0.f, 0.f, 0.f);
    if (norm) gv = *reinterpret_cast<const float4*>(rl + (nw - n0) + cg);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = g * 8 + hi * 4 + e;
          slab[r * 64 + l32] = acc[i][0][4 * g + e];
          slab[r * 64 + 32 + l32] = acc[i][1][4 * g + e];
        }
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int r = (lane >> 4) + 4 * k;
        const int64_t m = row_of(i, k);
        float ssq = 0.f;
        if (m < M) {
          const float4 sv = *reinterpret_cast<const float4*>(slab + r * 64 + cg);
          float4 xn = xo[k];
          xn.x += sv.x;
          xn.y += sv.y;
          xn.z += sv.z;
          xn.w += sv.w;
          *reinterpret_cast<float4*>(a.x + m * a.ldc + nw + cg) = xn;
          if (norm) {
            uint2 hv;
            hv.x = Op16<H>::cvt(xn.x * gv.x) | (static_cast<uint32_t>(Op16<H>::cvt(xn.y * gv.y)) << 16);
            hv.y = Op16<H>::cvt(xn.z * gv.z) | (static_cast<uint32_t>(Op16<H>::cvt(xn.w * gv.w)) << 16);
            *reinterpret_cast<uint2*>(hout + m * a.ldc + nw + cg) = hv;
            ssq = (xn.x * xn.x + xn.y * xn.y) + (xn.z * xn.z + xn.w * xn.w);
          }
        }
        if (norm) {
          ssq += __shfl_xor(ssq, 1);
          ssq += __shfl_xor(ssq, 2);
          ssq += __shfl_xor(ssq, 4);
          ssq += __shfl_xor(ssq, 8);
          if ((lane & 15) == 0 && m < M) a.ssp[m * a.n_part + part] = ssq;
        }
        if (i < 3) {   // the same row slot of the next slab
          int64_t mn = row_of(i + 1, k);
          if (mn > M - 1) mn = M - 1;
          if (EPI == EPI_RESID_EMB) {
            int32_t tok = a.x_tok[tok0 + mn];
            if (tok < 0 || tok >= a.vocab) tok = 0;
            const uint2 e = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(a.x_emb) +
                                                            static_cast<int64_t>(tok) * a.ldc + nw + cg);
            xo[k] = make_float4(Op16<H>::widen(static_cast<uint16_t>(e.x & 0xFFFFu)),
                                Op16<H>::widen(static_cast<uint16_t>(e.x >> 16)),
                                Op16<H>::widen(static_cast<uint16_t>(e.y & 0xFFFFu)),
                                Op16<H>::widen(static_cast<uint16_t>(e.y >> 16)));
          } else {
            xo[k] = *reinterpret_cast<const float4*>(a.x + mn * a.ldc + nw + cg);
          }
        }
      }
    }
    return;
  }
  prefetch();
  if (EPI == EPI_ARGMAX) {
    // row maxima over this wave's 64 columns: a row's values sit in the 32
    // lanes of one half-wave (column lane % 32, two 32-column blocks j); the
    // lanes meet in a butterfly that keeps the lower column on ties
    int2* P = static_cast<int2*>(a.C);
    const int chunk = nw >> 6;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float v = acc[i][0][4 * g + e];
          int c = nw + l32;
          const float v1 = acc[i][1][4 * g + e];
          if (v1 > v) {   // column + 32 only if strictly greater
            v = v1;
            c += 32;
          }
#pragma unroll
          for (int o = 1; o < 32; o <<= 1) {
            const float ov = __shfl_xor(v, o);
            const int oc = __shfl_xor(c, o);
            if (ov > v || (ov == v && oc < c)) {
              v = ov;
              c = oc;
            }
          }
          const int64_t m = mw + i * 32 + 8 * g + 4 * hi + e;
          if (l32 == 0 && m < M) P[m * a.ldc + chunk] = make_int2(__float_as_int(v), c);
        }
    return;
  }
  if (EPI == EPI_STORE_F32) {
    // fp32: four slabs of 32 rows x 64 columns (8 KB each)
    float* slab = reinterpret_cast<float*>(slice);
    float* C = static_cast<float*>(a.C);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = g * 8 + hi * 4 + e;
          slab[r * 64 + l32] = acc[i][0][4 * g + e];
          slab[r * 64 + 32 + l32] = acc[i][1][4 * g + e];
        }
      flush_slab<float>(slab, 32, 64, C, a.ldc, mw + i * 32, M, lane, [&](int c) { return nw + c; });
    }
    return;
  }
  // bf16 outputs: slab of 64 rows (two i-blocks) x 64 (or 32 for SwiGLU) columns
  uint16_t* C = static_cast<uint16_t*>(a.C);
  const bool is_v = EPI == EPI_QKV_ROPE && nw >= a.n_q + a.n_kv;
  int sbase = 0, head = 0, hh = 0, half = 0;
  float rev_per_pos = 0.f;
  if (EPI == EPI_QKV_ROPE && !is_v) {
    sbase = nw < a.n_q ? 0 : a.n_q;
    const int c = nw - sbase;
    head = c / a.hd;
    hh = (c % a.hd) >> 6;   // 0 except the second half-wave of a 128-dim head
    half = a.hd >> 1;
    // rotary frequency of this lane's lower-half dim, in revolutions per position
    rev_per_pos = hh ? rev.y : rev.x;
  }
  // q / k columns (rotary) or v columns: chosen once per wave (a per-element
  // choice costs exec-mask branches around every element)
  auto emit = [&](auto rot_tag) {
    constexpr bool ROT = decltype(rot_tag)::value;
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2) {
#pragma unroll
      for (int ii = 0; ii < 2; ++ii) {
        const int i = h2 * 2 + ii;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int tr = wm * 128 + i * 32 + g * 8 + hi * 4;   // tile row of e = 0
          int4 p4 = make_int4(0, 0, 0, 0);
          if (EPI == EPI_QKV_ROPE && ROT)   // positions of the 4 rows e = 0..3
            p4 = *reinterpret_cast<const int4*>(pl + tr);
          const int pe[4] = {p4.x, p4.y, p4.z, p4.w};
          float4 r4 = make_float4(1.f, 1.f, 1.f, 1.f);
          if (a.rs) r4 = *reinterpret_cast<const float4*>(rl + tr);   // RMSNorm row scales
          const float re[4] = {r4.x, r4.y, r4.z, r4.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int r = ii * 32 + g * 8 + hi * 4 + e;   // row inside the 64-row slab
            const float v0 = acc[i][0][4 * g + e] * re[e], v1 = acc[i][1][4 * g + e] * re[e];
            if (EPI == EPI_SWIGLU) {
              slice[r * 32 + l32] = Op16<H>::cvt(silu_fast(v0) * v1);
            } else if (EPI == EPI_QKV_ROPE && ROT) {
              // angle pos * theta^(-2i/hd), in revolutions (hardware sin/cos take revolutions)
              const float rev = static_cast<float>(pe[e]) * rev_per_pos;
              const float frac = rev - floorf(rev);
              const float cs = __builtin_amdgcn_cosf(frac), sn = __builtin_amdgcn_sinf(frac);
              slice[r * 64 + l32] = f2h(v0 * cs - v1 * sn);        // lower half dims
              slice[r * 64 + 32 + l32] = f2h(v1 * cs + v0 * sn);   // upper half dims
            } else if (EPI == EPI_QKV_ROPE && !ROT) {   // v
              slice[r * 64 + l32] = f2h(v0);
              slice[r * 64 + 32 + l32] = f2h(v1);
            } else {
              slice[r * 64 + l32] = Op16<H>::cvt(v0);
              slice[r * 64 + 32 + l32] = Op16<H>::cvt(v1);
            }
          }
        }
      }
      const int64_t m_first = mw + h2 * 64;
      if (EPI == EPI_SWIGLU) {
        flush_slab<uint16_t>(slice, 64, 32, C, a.ldc, m_first, M, lane, [&](int c) { return nw / 2 + c; });
      } else if (EPI == EPI_QKV_ROPE && ROT) {
        // slab columns 0..31: lower-half dims hh*32.., 32..63: the matching upper-half dims
        const int base = sbase + head * a.hd + hh * 32;
        flush_slab<uint16_t>(slice, 64, 64, C, a.ldc, m_first, M, lane,
                             [&](int c) { return base + (c < 32 ? c : half + c - 32); });
      } else {
        flush_slab<uint16_t>(slice, 64, 64, C, a.ldc, m_first, M, lane, [&](int c) { return nw + c; });
      }
    }
  };
  if (EPI == EPI_QKV_ROPE && !is_v)
    emit(std::true_type{});
  else
    emit(std::false_type{});
}

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// LDS stage: [256 rows][64 bf16], 128-byte rows of eight 16-byte chunks.  The
// chunk index is XORed with bits 1..3 of the row: 16 consecutive rows then
// cover all 64 banks once (row parity already picks the bank half).
__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }

// One 64-deep k-step of the wave's 128 x 64 sub-tile from one LDS stage.
// Fragments of the next 16-deep sub-step are read while the MFMAs of the
// current one run (two register sets), so LDS latency hides behind MFMA work.
template <bool H>
__device__ __forceinline__ void load_frags(const uint16_t* As, const uint16_t* Bs, int s, int wm, int wn, int lane,
                                           typename Op16<H>::V (&af)[4], typename Op16<H>::V (&bw)[2]) {
  typedef typename Op16<H>::V V;
  const int r32 = lane & 31;
  const int sw = swz(r32, 2 * s + (lane >> 5)) << 3;   // same for every 32-row block
#pragma unroll
  for (int i = 0; i < 4; ++i) af[i] = *reinterpret_cast<const V*>(As + (wm * 128 + i * 32 + r32) * GK + sw);
#pragma unroll
  for (int j = 0; j < 2; ++j) bw[j] = *reinterpret_cast<const V*>(Bs + (wn * 64 + j * 32 + r32) * GK + sw);
}

template <bool H>
__device__ __forceinline__ void mma_stage(const uint16_t* As, const uint16_t* Bs, f32x16 (&acc)[4][2], int wm,
                                          int wn, int lane) {
  typename Op16<H>::V af[2][4], bw[2][2];
  load_frags<H>(As, Bs, 0, wm, wn, lane, af[0], bw[0]);
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const int cur = s & 1;
    if (s < 3) load_frags<H>(As, Bs, s + 1, wm, wn, lane, af[cur ^ 1], bw[cur ^ 1]);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        acc[i][j] = Op16<H>::mma(af[cur][i], bw[cur][j], acc[i][j]);
    if (s < 3) {
      // interleave: one MFMA, one LDS read, ... then the remaining MFMAs
      for (int q = 0; q < 6; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // DS read
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    }
  }
}

// Global -> LDS tile copy with the 16-byte direct-to-LDS load: a wave's
// instruction fills 1 KB (8 rows) at consecutive lane slots, so lane l
// fetches the global chunk that belongs at row 8c + l/8, slot l%8.
__device__ __forceinline__ void dma_stage(uint16_t* sA, uint16_t* sB, const uint16_t* const (&ga)[4],
                                          const uint16_t* const (&gb)[4], int k0, int w) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = i * 8 + w;
    __builtin_amdgcn_global_load_lds(static_cast<const void*>(ga[i] + k0), (lds_ptr_t)(sA + c * 512), 16, 0, 0);
    __builtin_amdgcn_global_load_lds(static_cast<const void*>(gb[i] + k0), (lds_ptr_t)(sB + c * 512), 16, 0, 0);
  }
}

template <int EPI>
__device__ __forceinline__ void tile_sources(const GemmArgs& a, const uint16_t* A, int64_t M, int64_t m0, int n0,
                                             int w, int lane, const uint16_t* (&ga)[4], const uint16_t* (&gb)[4]) {
  const int lr = lane >> 3;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = (i * 8 + w) * 8 + lr;
    const int lc = swz(row, lane & 7);   // logical chunk stored in this lane's slot
    int64_t mr = m0 + row;
    if (mr > M - 1) mr = M - 1;
    ga[i] = A + mr * a.lda + lc * 8;
    gb[i] = b_row<EPI, uint16_t>(a, n0 + row) + lc * 8;
  }
}

template <int EPI, bool H>
__global__ __launch_bounds__(GT) void k_gemm_bf16(GemmArgs a) {
  // two stages in distinct arrays: the compiler can then tell the in-flight
  // loads into one stage from the reads of the other and only waits at the
  // barrier that ends the stage
  __shared__ __attribute__((aligned(16))) uint16_t sA0[GM * GK];
  __shared__ __attribute__((aligned(16))) uint16_t sB0[GN * GK];
  __shared__ __attribute__((aligned(16))) uint16_t sA1[GM * GK];
  __shared__ __attribute__((aligned(16))) uint16_t sB1[GN * GK];
  __shared__ __attribute__((aligned(16))) float rbuf[GM];     // the tile's RMSNorm row scales
  __shared__ __attribute__((aligned(16))) int32_t pbuf[GM];   // the tile's token positions (QKV)
  const int64_t M = *a.m_ptr;
  if (M <= 0) return;
  const int tiles_n = a.N / GN;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6, wm = w >> 2, wn = w & 3;
  const int nk = a.K / GK;
  const uint16_t* A = static_cast<const uint16_t*>(a.A);

  // XCD-aware order: workgroups are dispatched round-robin over the 8 XCDs,
  // so workgroup b runs on XCD b % 8.  XCD x owns the M-tile rows
  // tm = x, x + 8, x + 16, ...; inside an XCD the tiles go in groups of
  // GROUP_M of its rows, column by column, so the 32 workgroups resident on
  // one XCD share a few activation row-panels and a few weight column-panels
  // in that XCD's L2 instead of streaming 32 distinct panels.
  constexpr int GROUP_M = 4;
  const int64_t tiles_m = (M + GM - 1) / GM;
  const int xcd = blockIdx.x & 7;
  const int64_t per_xcd = gridDim.x >> 3;   // grid is a multiple of 8
  const int64_t rows_x = tiles_m > xcd ? (tiles_m - xcd + 7) / 8 : 0;
  const int64_t count_x = rows_x * tiles_n;
  auto tile_mn = [&](int64_t q, int64_t& m0, int& n0) {
    const int64_t per_group = static_cast<int64_t>(GROUP_M) * tiles_n;
    const int64_t grp = q / per_group, within = q % per_group;
    const int64_t rows_here = (rows_x - grp * GROUP_M) < GROUP_M ? (rows_x - grp * GROUP_M) : GROUP_M;
    const int64_t lr = grp * GROUP_M + within % rows_here;
    m0 = (lr * 8 + xcd) * GM;
    n0 = static_cast<int>(within / rows_here) * GN;
  };
  int64_t q = blockIdx.x >> 3;
  if (q >= count_x) return;
  float2 rev = make_float2(0.f, 0.f);
  if (EPI == EPI_QKV_ROPE) {
    const int l32 = lane & 31;
    rev.x = a.rope_rev[l32];
    if (a.hd == 128) rev.y = a.rope_rev[32 + l32];
  }
  const uint16_t* ga[4];
  const uint16_t* gb[4];
  {
    int64_t m0;
    int n0;
    tile_mn(q, m0, n0);
    tile_sources<EPI>(a, A, M, m0, n0, w, lane, ga, gb);
  }
  dma_stage(sA0, sB0, ga, gb, 0, w);
  for (; q < count_x; q += per_xcd) {
    int64_t m0;
    int n0;
    tile_mn(q, m0, n0);
    f32x16 acc[4][2];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;
    __syncthreads();   // stage 0 of this tile has landed; the last epilogue is done with rbuf / pbuf
    // the tile's row scales and positions go to LDS now, so that the epilogue
    // reads no global memory behind the next tile's prefetch
    if (w == 0 && (EPI == EPI_QKV_ROPE || EPI == EPI_SWIGLU) && a.rs)
      __builtin_amdgcn_global_load_lds(static_cast<const void*>(a.rs + m0 + lane * 4), (lds_ptr_t)(rbuf + lane * 4),
                                       16, 0, 0);
    if (w == 0 && (EPI == EPI_RESID || EPI == EPI_RESID_EMB) && a.gnext)   // the following norm's gain for the tile's columns
      __builtin_amdgcn_global_load_lds(static_cast<const void*>(a.gnext + n0 + lane * 4),
                                       (lds_ptr_t)(rbuf + lane * 4), 16, 0, 0);
    if (w == 1 && EPI == EPI_QKV_ROPE)
      __builtin_amdgcn_global_load_lds(static_cast<const void*>(a.pos + m0 + lane * 4), (lds_ptr_t)(pbuf + lane * 4),
                                       16, 0, 0);
    for (int kt = 0; kt < nk; kt += 2) {
      if (kt + 1 < nk) dma_stage(sA1, sB1, ga, gb, (kt + 1) * GK, w);
      mma_stage<H>(sA0, sB0, acc, wm, wn, lane);
      __syncthreads();
      if (kt + 1 < nk) {
        if (kt + 2 < nk) dma_stage(sA0, sB0, ga, gb, (kt + 2) * GK, w);
        mma_stage<H>(sA1, sB1, acc, wm, wn, lane);
        __syncthreads();
      }
    }
    // stage 0 is free: the next tile's first k-step loads under the epilogue
    const bool more = q + per_xcd < count_x;
    auto prefetch = [&]() {
      if (more) {
        int64_t m1;
        int n1;
        tile_mn(q + per_xcd, m1, n1);
        tile_sources<EPI>(a, A, M, m1, n1, w, lane, ga, gb);
        dma_stage(sA0, sB0, ga, gb, 0, w);
      }
    };
    // each wave stages its output in its own 8 KB slice of stage 1, which is
    // idle until the next tile's first barrier
    uint16_t* slice = (w < 4 ? sA1 : sB1) + (w & 3) * 4096;
    epilogue_bf16<EPI, H>(a, acc, m0, n0, M, wm, wn, lane, slice, rbuf, pbuf, rev, prefetch);
  }
}

hipError_t launch_gemm_bf16(int epi, const GemmArgs& a, hipStream_t s) {
  // one workgroup per CU, rounded to whole XCD groups; fewer for small problems
  const int64_t tiles = ((a.m_ub + GM - 1) / GM) * (a.N / GN);
  int64_t g = num_cus();
  if (tiles < g) g = tiles;
  g = (g + 7) / 8 * 8;
  const dim3 grid(static_cast<unsigned>(g)), block(GT);
#define AIQ_LAUNCH_GEMM(E)                                                         \
  do {                                                                             \
    if (a.f16)                                                                     \
      hipLaunchKernelGGL((k_gemm_bf16<E, true>), grid, block, 0, s, a);            \
    else                                                                           \
      hipLaunchKernelGGL((k_gemm_bf16<E, false>), grid, block, 0, s, a);           \
  } while (0)
  switch (epi) {
    case EPI_STORE_F32: AIQ_LAUNCH_GEMM(EPI_STORE_F32); break;
    case EPI_ARGMAX:
      if (a.ldc != a.N / 64) return hipErrorInvalidValue;
      AIQ_LAUNCH_GEMM(EPI_ARGMAX);
      break;
    case EPI_STORE_ACT: AIQ_LAUNCH_GEMM(EPI_STORE_ACT); break;
    case EPI_SWIGLU: AIQ_LAUNCH_GEMM(EPI_SWIGLU); break;
    case EPI_QKV_ROPE: AIQ_LAUNCH_GEMM(EPI_QKV_ROPE); break;
    case EPI_RESID:
    case EPI_RESID_EMB:
      if (a.ldc != a.N || a.N % 64 || (a.gnext && (!a.hout || !a.ssp || a.n_part != a.N / 64)))
        return hipErrorInvalidValue;
      if (epi == EPI_RESID_EMB) {
        if (!a.x_emb || !a.x_tok || !a.x_tok_desc || a.vocab <= 0) return hipErrorInvalidValue;
        AIQ_LAUNCH_GEMM(EPI_RESID_EMB);
      } else {
        AIQ_LAUNCH_GEMM(EPI_RESID);
      }
      break;
    default: return hipErrorInvalidValue;
  }
#undef AIQ_LAUNCH_GEMM
  return hipGetLastError();
}

// ======================================================================= fp32 FMA
constexpr int FM = 64, FN = 64, FK = 16, FT = 256;

template <int EPI>
__global__ __launch_bounds__(FT) void k_gemm_f32(GemmArgs a) {
  __shared__ float As[FK][FM + 4];
  __shared__ float Bs[FK][FN + 4];
  const int64_t M = *a.m_ptr;
  if (M <= 0) return;
  const int tiles_n = a.N / FN;
  const int64_t n_tiles = ((M + FM - 1) / FM) * tiles_n;
  const int t = threadIdx.x, ty = t >> 4, tx = t & 15;
  const float* A = static_cast<const float*>(a.A);
  const int lrow = t >> 2, lk = (t & 3) * 4;
  for (int64_t tile = blockIdx.x; tile < n_tiles; tile += gridDim.x) {
    const int64_t m0 = (tile / tiles_n) * FM;
    const int n0 = static_cast<int>(tile % tiles_n) * FN;
    int64_t mr = m0 + lrow;
    if (mr > M - 1) mr = M - 1;
    const float* ap = A + mr * a.lda + lk;
    const float* bp = b_row<EPI, float>(a, n0 + lrow) + lk;
    float acc[4][4] = {};
    for (int k0 = 0; k0 < a.K; k0 += FK) {
      const float4 av = *reinterpret_cast<const float4*>(ap + k0);
      const float4 bv = *reinterpret_cast<const float4*>(bp + k0);
      __syncthreads();
      As[lk + 0][lrow] = av.x; As[lk + 1][lrow] = av.y; As[lk + 2][lrow] = av.z; As[lk + 3][lrow] = av.w;
      Bs[lk + 0][lrow] = bv.x; Bs[lk + 1][lrow] = bv.y; Bs[lk + 2][lrow] = bv.z; Bs[lk + 3][lrow] = bv.w;
      __syncthreads();
#pragma unroll
      for (int k = 0; k < FK; ++k) {
        float ar[4], br[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          ar[i] = As[k][ty * 4 + i];
          br[i] = Bs[k][tx * 4 + i];
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(ar[i], br[j], acc[i][j]);
      }
    }
    const int n = n0 + tx * 4;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t m = m0 + ty * 4 + i;
      if (m >= M) continue;
      if (EPI == EPI_GELU) {
        *reinterpret_cast<float4*>(static_cast<float*>(a.C) + m * a.ldc + n) =
            make_float4(gelu_erf(acc[i][0]), gelu_erf(acc[i][1]), gelu_erf(acc[i][2]), gelu_erf(acc[i][3]));
      } else {  // plain fp32 store (QKV columns in natural order; rotary applied afterwards)
        *reinterpret_cast<float4*>(static_cast<float*>(a.C) + m * a.ldc + n) =
            make_float4(acc[i][0], acc[i][1], acc[i][2], acc[i][3]);
      }
    }
  }
}

hipError_t launch_gemm_f32(int epi, const GemmArgs& a, hipStream_t s) {
  const int64_t tiles = ((a.m_ub + FM - 1) / FM) * (a.N / FN);
  int64_t g = static_cast<int64_t>(num_cus()) * 4;
  if (tiles < g) g = tiles;
  if (g < 1) g = 1;
  const dim3 grid(static_cast<unsigned>(g)), block(FT);
  switch (epi) {
    case EPI_STORE_F32:
    case EPI_STORE_ACT: hipLaunchKernelGGL(k_gemm_f32<EPI_STORE_F32>, grid, block, 0, s, a); break;
    case EPI_QKV_ROPE: hipLaunchKernelGGL(k_gemm_f32<EPI_QKV_ROPE>, grid, block, 0, s, a); break;
    case EPI_GELU: hipLaunchKernelGGL(k_gemm_f32<EPI_GELU>, grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Rotary embedding in place on the q and k columns of an fp32 QKV buffer.
__global__ void k_rope_f32(const int64_t* desc, float* qkv, int64_t ld, int32_t n_q, int32_t n_kv, int32_t hd,
                           const int32_t* pos, const float* cos_t, const float* sin_t) {
  const int64_t nt = desc[D_NTOK];
  const int half = hd >> 1;
  const int heads = (n_q + n_kv) / hd;
  const int64_t total = nt * heads * half;
  for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < total; j += (int64_t)gridDim.x * blockDim.x) {
    const int i = static_cast<int>(j % half);
    const int64_t th = j / half;
    const int h = static_cast<int>(th % heads);
    const int64_t t = th / heads;
    float* base = qkv + t * ld + static_cast<int64_t>(h) * hd;   // q heads then k heads are contiguous
    const int64_t ti = static_cast<int64_t>(pos[t]) * half + i;
    const float c = cos_t[ti], s = sin_t[ti];
    const float x1 = base[i], x2 = base[i + half];
    base[i] = x1 * c - x2 * s;
    base[i + half] = x2 * c + x1 * s;
  }
}

hipError_t launch_rope_f32(const int64_t* desc, float* qkv, int64_t ld, int32_t n_q, int32_t n_kv,
                           int32_t hd, const int32_t* pos, const float* cos_t, const float* sin_t,
                           int64_t t_cap, hipStream_t s) {
  int64_t g = (t_cap * ((n_q + n_kv) / hd) * (hd / 2) + 255) / 256;
  if (g > 4096) g = 4096;
  if (g < 1) g = 1;
  hipLaunchKernelGGL(k_rope_f32, dim3(static_cast<unsigned>(g)), dim3(256), 0, s, desc, qkv, ld, n_q, n_kv, hd,
                     pos, cos_t, sin_t);
  return hipGetLastError();
}

}  // namespace aiq
