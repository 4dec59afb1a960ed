// Dense projections of the prefill: C[M, N] = A[M, K] . W[N, K]^T with fused
// epilogues (rotary embedding on q/k, SwiGLU, GELU, residual add).
//
// bf16 / fp16 path (gfx950 MFMA): 256 x 256 output tile per 256-thread
// workgroup (one per CU), K stepped by 64 through two LDS stages (2 x 64 KB)
// filled by 16-byte direct-to-LDS loads.  Four waves, one per SIMD, in a
// 2 x 2 grid each own a 128 x 128 sub-tile = 4 x 4 blocks of
// v_mfma_f32_32x32x16 (256 accumulator registers per lane).  The next
// stage's loads are spread over the MFMAs of the first three quarters of the
// current one (a burst of them stalls the wave's MFMA issue), and each wave's loads
// go to 4 KB-contiguous LDS runs so one M0 value serves four of them through
// the instruction's immediate offset.  The next tile's first stage is
// fetched while the epilogue of the current one runs.
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
  if (hd != 128) return c;   // 64-dim heads: natural order
  const int head = c >> 7, cc = c & 127;
  const int hh = cc >> 6, jj = cc & 63;
  const int dim = jj < 32 ? hh * 32 + jj : 64 + hh * 32 + (jj - 32);
  return head * 128 + dim;
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
constexpr int GM = 256, GN = 256, GK = 64, GT = 256;

typedef f32x16_t f32x16;

// Accumulator layout.  The MFMAs compute the transposed tile, weights as the
// first operand (v_mfma_f32_32x32x16: D[r][c] with r = 8g + 4*(lane/32) + e
// in register 4g + e, c = lane % 32): acc[i][j][4g + e] holds C[m][n] with
//   m = m0 + wm*128 + i*32 + lane%32,   n = n0 + wn*128 + j*32 + 8g + 4*(lane/32) + e,
// four consecutive columns of one row per (j, g).
//
// Epilogue: for each 32-row block i the wave writes its 32 x 128 fp32
// accumulators to its own 16 KB slice of the idle LDS stage, 16 bytes per
// (j, g) straight from the accumulator registers, then reads them back as
// pieces of 8 consecutive columns of one row, 16 consecutive lanes covering
// one row, so every global access of the epilogue is a contiguous run of
// 256 or 512 bytes per row.  The SwiGLU pair (columns c and c + 32 of a
// 64-column half: gate and up) and the rotary pair (lower and upper half of
// a head's dims, as the q/k weight rows are reordered) are pieces 4 apart.
//
// q, k and v (attention operands) are stored in fp16: 10 mantissa bits where
// bf16 has 7, at the same MFMA rate; their magnitudes are O(1) after RMSNorm.

// Lane exchange through a DPP move (a VALU op; a lane shuffle goes through
// the LDS crossbar).  The residual epilogue's butterfly takes the same
// partners and adds in the same order as lane ^ 1, ^ 2, ^ 4 shuffles: after
// the first two steps the four lanes of a quad hold equal sums, so the
// mirrored quad is the ^ 4 partner's.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, false));
}

__device__ __forceinline__ float silu_fast(float g) {
  return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g));
}

template <bool H>
__device__ __forceinline__ uint4 pack8(const float (&v)[8]) {
  uint4 p;
  p.x = Op16<H>::cvt(v[0]) | (static_cast<uint32_t>(Op16<H>::cvt(v[1])) << 16);
  p.y = Op16<H>::cvt(v[2]) | (static_cast<uint32_t>(Op16<H>::cvt(v[3])) << 16);
  p.z = Op16<H>::cvt(v[4]) | (static_cast<uint32_t>(Op16<H>::cvt(v[5])) << 16);
  p.w = Op16<H>::cvt(v[6]) | (static_cast<uint32_t>(Op16<H>::cvt(v[7])) << 16);
  return p;
}
__device__ __forceinline__ uint4 pack8h(const float (&v)[8]) {
  uint4 p;
  p.x = f2h(v[0]) | (static_cast<uint32_t>(f2h(v[1])) << 16);
  p.y = f2h(v[2]) | (static_cast<uint32_t>(f2h(v[3])) << 16);
  p.z = f2h(v[4]) | (static_cast<uint32_t>(f2h(v[5])) << 16);
  p.w = f2h(v[6]) | (static_cast<uint32_t>(f2h(v[7])) << 16);
  return p;
}

// The wave's epilogue slice: 32 rows x 128 fp32, 512-byte rows of 32
// 16-byte chunks; chunk c of row r sits at slot c ^ (r & 15), so 16
// consecutive rows writing one chunk, and one row read by 16 lanes, each
// cover all 64 banks.
__device__ __forceinline__ int eslot(int r, int c) { return r * 32 + (c ^ (r & 15)); }

// Makes this wave's LDS writes visible to its own later reads in other
// lanes (LDS completes one wave's operations in order; this keeps the
// compiler from moving them across).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// `rl` holds the tile's row scales (QKV, SwiGLU) or the following norm's gain
// for the tile's columns (residual), `pl` the tile's positions and `rv` the
// rotary frequencies of a head's lower-half dims (revolutions per position),
// all in LDS; `slice` is the wave's 16 KB of idle LDS.  `prefetch` issues the
// next tile's first loads (after the residual epilogue's first loads of x,
// so that those do not queue behind it; first for the others).
template <int EPI, bool H, typename Prefetch>
__device__ __forceinline__ void epilogue_bf16(const GemmArgs& a, f32x16 (&acc)[4][4], int64_t m0, int n0,
                                              int64_t M, int wm, int wn, int lane, float4* slice, const float* rl,
                                              const int32_t* pl, const float* rv, Prefetch prefetch) {
  const int l32 = lane & 31, hi = lane >> 5;
  const int nw = n0 + wn * 128;   // first GEMM column of the wave's sub-tile
  const int pc = lane & 15;       // piece (8 columns) of a row this lane reads back
  const int pr = lane >> 4;       // its row inside each group of 4 rows
  constexpr bool RESID = EPI == EPI_RESID || EPI == EPI_RESID_EMB;
  if (!RESID) prefetch();
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    // fp32 accumulators of rows 32i .. 32i + 31 to LDS
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        slice[eslot(l32, 8 * j + 2 * g + hi)] =
            make_float4(acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]);
    wave_lds_sync();
    const int row0 = wm * 128 + i * 32;   // tile row of slice row 0
    if (RESID) {
      // x += acc in place; with a following norm also h = x * g and, per row,
      // the sum of x^2 over each 64-column half (pieces 8h .. 8h + 7, eight
      // neighbouring lanes, added in a fixed butterfly order).  All eight
      // rows' residuals of this lane are read before any is used.
      const bool norm = a.gnext != nullptr;
      uint16_t* hout = static_cast<uint16_t*>(a.hout);
      const int64_t tok0 = EPI == EPI_RESID_EMB ? a.x_tok_desc[D_TOK_BEGIN] : 0;
      const int col = nw + 8 * pc;
      float4 xv[8][2];
#pragma unroll
      for (int rr = 0; rr < 8; ++rr) {
        int64_t m = m0 + row0 + 4 * rr + pr;
        if (m > M - 1) m = M - 1;   // in bounds; the value is not used
        if (EPI == EPI_RESID_EMB) {
          // the residual before this projection is the token's embedding row
          // widened from 16 bits, which is exactly what x would hold
          int32_t tok = a.x_tok[tok0 + m];
          if (tok < 0 || tok >= a.vocab) tok = 0;
          const uint4 e = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(a.x_emb) +
                                                          static_cast<int64_t>(tok) * a.ldc + col);
          xv[rr][0] = make_float4(Op16<H>::widen(static_cast<uint16_t>(e.x & 0xFFFFu)),
                                  Op16<H>::widen(static_cast<uint16_t>(e.x >> 16)),
                                  Op16<H>::widen(static_cast<uint16_t>(e.y & 0xFFFFu)),
                                  Op16<H>::widen(static_cast<uint16_t>(e.y >> 16)));
          xv[rr][1] = make_float4(Op16<H>::widen(static_cast<uint16_t>(e.z & 0xFFFFu)),
                                  Op16<H>::widen(static_cast<uint16_t>(e.z >> 16)),
                                  Op16<H>::widen(static_cast<uint16_t>(e.w & 0xFFFFu)),
                                  Op16<H>::widen(static_cast<uint16_t>(e.w >> 16)));
        } else {
          const float* xr = a.x + m * a.ldc + col;
          xv[rr][0] = *reinterpret_cast<const float4*>(xr);
          xv[rr][1] = *reinterpret_cast<const float4*>(xr + 4);
        }
      }
      if (i == 0) prefetch();
      float4 g0 = make_float4(0.f, 0.f, 0.f, 0.f), g1 = g0;
      if (norm) {
        g0 = *reinterpret_cast<const float4*>(rl + (col - n0));
        g1 = *reinterpret_cast<const float4*>(rl + (col - n0) + 4);
      }
#pragma unroll
      for (int rr = 0; rr < 8; ++rr) {
        const int r = 4 * rr + pr;
        const int64_t m = m0 + row0 + r;
        const float4 s0 = slice[eslot(r, 2 * pc)], s1 = slice[eslot(r, 2 * pc + 1)];
        float4 x0 = xv[rr][0], x1 = xv[rr][1];
        x0.x += s0.x; x0.y += s0.y; x0.z += s0.z; x0.w += s0.w;
        x1.x += s1.x; x1.y += s1.y; x1.z += s1.z; x1.w += s1.w;
        float ssq = 0.f;
        if (m < M) {
          float* xr = a.x + m * a.ldc + col;
          *reinterpret_cast<float4*>(xr) = x0;
          *reinterpret_cast<float4*>(xr + 4) = x1;
          if (norm) {
            const float hv[8] = {x0.x * g0.x, x0.y * g0.y, x0.z * g0.z, x0.w * g0.w,
                                 x1.x * g1.x, x1.y * g1.y, x1.z * g1.z, x1.w * g1.w};
            *reinterpret_cast<uint4*>(hout + m * a.ldc + col) = pack8<H>(hv);
          }
          ssq = ((x0.x * x0.x + x0.y * x0.y) + (x0.z * x0.z + x0.w * x0.w)) +
                ((x1.x * x1.x + x1.y * x1.y) + (x1.z * x1.z + x1.w * x1.w));
        }
        if (norm) {
          ssq += dpp_f32<0xB1>(ssq);    // quad_perm [1,0,3,2]: lane ^ 1
          ssq += dpp_f32<0x4E>(ssq);    // quad_perm [2,3,0,1]: lane ^ 2
          ssq += dpp_f32<0x141>(ssq);   // row_half_mirror: the other quad of the eight, whose lanes agree
          if ((pc & 7) == 0 && m < M) a.ssp[m * a.n_part + ((nw >> 6) + (pc >> 3))] = ssq;
        }
      }
    } else if (EPI == EPI_ARGMAX) {
      // row maxima over each 64-column half: the lane's 8 columns in
      // increasing order (a strictly greater value replaces), then the eight
      // lanes of the half in a butterfly that keeps the lower column on ties
      int2* P = static_cast<int2*>(a.C);
#pragma unroll
      for (int rr = 0; rr < 8; ++rr) {
        const int r = 4 * rr + pr;
        const int64_t m = m0 + row0 + r;
        const float4 s0 = slice[eslot(r, 2 * pc)], s1 = slice[eslot(r, 2 * pc + 1)];
        const float v8[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
        float v = v8[0];
        int c = nw + 8 * pc;
#pragma unroll
        for (int e = 1; e < 8; ++e)
          if (v8[e] > v) {
            v = v8[e];
            c = nw + 8 * pc + e;
          }
#pragma unroll
        for (int o = 1; o < 8; o <<= 1) {
          const float ov = __shfl_xor(v, o);
          const int oc = __shfl_xor(c, o);
          if (ov > v || (ov == v && oc < c)) {
            v = ov;
            c = oc;
          }
        }
        if ((pc & 7) == 0 && m < M) P[m * a.ldc + ((nw >> 6) + (pc >> 3))] = make_int2(__float_as_int(v), c);
      }
    } else if (EPI == EPI_STORE_F32) {
      float* C = static_cast<float*>(a.C);
#pragma unroll
      for (int rr = 0; rr < 8; ++rr) {
        const int r = 4 * rr + pr;
        const int64_t m = m0 + row0 + r;
        if (m < M) {
          float* cr = C + m * a.ldc + nw + 8 * pc;
          *reinterpret_cast<float4*>(cr) = slice[eslot(r, 2 * pc)];
          *reinterpret_cast<float4*>(cr + 4) = slice[eslot(r, 2 * pc + 1)];
        }
      }
    } else if (EPI == EPI_STORE_ACT) {
      uint16_t* C = static_cast<uint16_t*>(a.C);
#pragma unroll
      for (int rr = 0; rr < 8; ++rr) {
        const int r = 4 * rr + pr;
        const int64_t m = m0 + row0 + r;
        const float4 s0 = slice[eslot(r, 2 * pc)], s1 = slice[eslot(r, 2 * pc + 1)];
        const float v8[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
        if (m < M) *reinterpret_cast<uint4*>(C + m * a.ldc + nw + 8 * pc) = pack8<H>(v8);
      }
    } else {
      // SwiGLU and rotary pairs: pieces q (0..3) and q + 4 of one 64-column
      // half h; lane piece pc -> (h, q) = (pc / 8, pc % 4) on rows of parity
      // pc / 4 % 2: 32 rows x 2 halves x 4 pairs = 256 pair-pieces, 4 per lane
      uint16_t* C = static_cast<uint16_t*>(a.C);
      const int h = pc >> 3, q = pc & 3, rp = (pc >> 2) & 1;
      const int nh = nw + 64 * h;
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int r = 8 * rr + 2 * pr + rp;
        const int tr = row0 + r;
        const int64_t m = m0 + tr;
        const float rs = a.rs ? rl[tr] : 1.f;   // RMSNorm row scale
        const float4 l0 = slice[eslot(r, 16 * h + 2 * q)], l1 = slice[eslot(r, 16 * h + 2 * q + 1)];
        const float4 u0 = slice[eslot(r, 16 * h + 2 * q + 8)], u1 = slice[eslot(r, 16 * h + 2 * q + 9)];
        const float lo[8] = {l0.x * rs, l0.y * rs, l0.z * rs, l0.w * rs, l1.x * rs, l1.y * rs, l1.z * rs, l1.w * rs};
        const float up[8] = {u0.x * rs, u0.y * rs, u0.z * rs, u0.w * rs, u1.x * rs, u1.y * rs, u1.z * rs, u1.w * rs};
        if (m >= M) continue;
        uint16_t* crow = C + m * a.ldc;
        if (EPI == EPI_SWIGLU) {
          float o[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) o[e] = silu_fast(lo[e]) * up[e];
          *reinterpret_cast<uint4*>(crow + (nh >> 1) + 8 * q) = pack8<H>(o);
        } else if (nh >= a.n_q + a.n_kv) {   // v: natural order
          *reinterpret_cast<uint4*>(crow + nh + 8 * q) = pack8h(lo);
          *reinterpret_cast<uint4*>(crow + nh + 32 + 8 * q) = pack8h(up);
        } else {
          const int sbase = nh < a.n_q ? 0 : a.n_q;
          const int cc = nh - sbase;
          const int head = cc / a.hd, hh = (cc % a.hd) >> 6, half = a.hd >> 1;
          const float pos = static_cast<float>(pl[tr]);
          const float4 f0 = *reinterpret_cast<const float4*>(rv + hh * 32 + 8 * q);
          const float4 f1 = *reinterpret_cast<const float4*>(rv + hh * 32 + 8 * q + 4);
          const float fr[8] = {f0.x, f0.y, f0.z, f0.w, f1.x, f1.y, f1.z, f1.w};
          float ol[8], ou[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            // angle pos * theta^(-2i/hd), in revolutions (hardware sin/cos take revolutions)
            const float rev = pos * fr[e];
            const float frac = rev - floorf(rev);
            const float cs = __builtin_amdgcn_cosf(frac), sn = __builtin_amdgcn_sinf(frac);
            ol[e] = lo[e] * cs - up[e] * sn;   // lower half dim
            ou[e] = up[e] * cs + lo[e] * sn;   // upper half dim
          }
          uint16_t* dst = crow + sbase + head * a.hd + hh * 32 + 8 * q;
          *reinterpret_cast<uint4*>(dst) = pack8h(ol);
          *reinterpret_cast<uint4*>(dst + half) = pack8h(ou);
        }
      }
    }
    wave_lds_sync();   // the slice's reads are done before the next block's writes
  }
}

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// LDS stage: [256 rows][64 bf16], 128-byte rows of eight 16-byte chunks.  The
// chunk index is XORed with bits 1..3 of the row: 16 consecutive rows then
// cover all 64 banks once (row parity already picks the bank half).
__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }

// Fragments of one 16-deep sub-step s of the wave's 128 x 128 sub-tile.
template <bool H>
__device__ __forceinline__ void load_frags(const uint16_t* As, const uint16_t* Bs, int s, int wm, int wn, int lane,
                                           typename Op16<H>::V (&af)[4], typename Op16<H>::V (&bw)[4]) {
  typedef typename Op16<H>::V V;
  const int r32 = lane & 31;
  const int sw = swz(r32, 2 * s + (lane >> 5)) << 3;   // same for every 32-row block
#pragma unroll
  for (int i = 0; i < 4; ++i) af[i] = *reinterpret_cast<const V*>(As + (wm * 128 + i * 32 + r32) * GK + sw);
#pragma unroll
  for (int j = 0; j < 4; ++j) bw[j] = *reinterpret_cast<const V*>(Bs + (wn * 128 + j * 32 + r32) * GK + sw);
}

// 16-byte direct-to-LDS load whose immediate offset, (i % 4) KB, is added to
// both the global and the LDS address (the global pointer carries -(i % 4) KB).
__device__ __forceinline__ void load_lds_imm(const void* g, lds_ptr_t l, int i) {
  switch (i & 3) {
    case 0: __builtin_amdgcn_global_load_lds(g, l, 16, 0, 0); break;
    case 1: __builtin_amdgcn_global_load_lds(g, l, 16, 1024, 0); break;
    case 2: __builtin_amdgcn_global_load_lds(g, l, 16, 2048, 0); break;
    default: __builtin_amdgcn_global_load_lds(g, l, 16, 3072, 0); break;
  }
}

// Global -> LDS copy of one stage: wave w fills rows 64w .. 64w + 63 of A and
// of W (eight 1 KB pieces of 8 rows each); in a piece's instruction lane l
// fetches the global chunk that belongs at row 8c + l/8, slot l%8.  The
// source pointers advance by one k-step.
__device__ __forceinline__ void dma_stage(uint16_t* sA, uint16_t* sB, const uint16_t* (&ga)[8],
                                          const uint16_t* (&gb)[8], int w) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int c = 8 * w + (i & 4);
    load_lds_imm(static_cast<const void*>(ga[i]), (lds_ptr_t)(sA + c * 512), i);
    load_lds_imm(static_cast<const void*>(gb[i]), (lds_ptr_t)(sB + c * 512), i);
    ga[i] += GK;
    gb[i] += GK;
  }
}

// One 64-deep k-step of the wave's sub-tile from one LDS stage (4 sub-steps of
// 16 MFMAs).  Fragments of the next sub-step are read while the MFMAs of the
// current one run, and the next stage's 16 loads (8 pieces of A, then 8 of
// W) go out during the first three sub-steps, 5, 5 and 6 of them, each after
// an MFMA.  Issued over two sub-steps, the loads back up in the memory
// pipeline and stall MFMA issue on large problems (4 % slower at 2M rows);
// issued over all four, the last ones are still in flight at the stage's
// closing barrier.  The source pointers point at the k-block after the one
// being consumed; `dma` is false in the tile's last stage, when they are one
// past the row's end.  The loads then re-read the row's last k-block into the
// idle stage and the pointers stay, so every stage runs the same
// straight-line schedule (a branch around the loads splits the stage into
// blocks that the scheduler cannot interleave: 1-2 % slower).
template <bool H>
__device__ __forceinline__ void mma_stage(const uint16_t* As, const uint16_t* Bs, f32x16 (&acc)[4][4], int wm,
                                          int wn, int lane, uint16_t* nA, uint16_t* nB, const uint16_t* (&ga)[8],
                                          const uint16_t* (&gb)[8], int w, bool dma) {
  typename Op16<H>::V af[2][4], bw[2][4];
  load_frags<H>(As, Bs, 0, wm, wn, lane, af[0], bw[0]);
  __builtin_amdgcn_sched_barrier(0);   // the first sub-step's reads are not interleaved with its own MFMAs
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const int cur = s & 1;
    if (s < 3) load_frags<H>(As, Bs, s + 1, wm, wn, lane, af[cur ^ 1], bw[cur ^ 1]);
    const int l0 = (16 * s) / 3, l1 = s < 3 ? (16 * (s + 1)) / 3 : l0;   // this sub-step's loads [l0, l1)
    const int back = dma ? 0 : -GK, adv = dma ? GK : 0;
#pragma unroll
    for (int l = l0; l < l1; ++l) {
      const int i = l & 7, c = 8 * w + (i & 4);
      if (l < 8) {
        load_lds_imm(static_cast<const void*>(ga[i] + back), (lds_ptr_t)(nA + c * 512), i);
        ga[i] += adv;
      } else {
        load_lds_imm(static_cast<const void*>(gb[i] + back), (lds_ptr_t)(nB + c * 512), i);
        gb[i] += adv;
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = Op16<H>::mma(bw[cur][j], af[cur][i], acc[i][j]);
    // the first 8 MFMAs each followed by one fragment read and (while any
    // are left) one load, then the other 8
    for (int q = 0; q < 8; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                  // MFMA
      if (s < 3) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);       // DS read
      if (q < l1 - l0) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0); // VMEM read
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
    __builtin_amdgcn_sched_barrier(0);
  }
}

// Source pointers of a tile's first k-step (see dma_stage), each carrying
// -(i % 4) KB for the loads' immediate offset.
template <int EPI>
__device__ __forceinline__ void tile_sources(const GemmArgs& a, const uint16_t* A, int64_t M, int64_t m0, int n0,
                                             int w, int lane, const uint16_t* (&ga)[8], const uint16_t* (&gb)[8]) {
  const int lr = lane >> 3;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int row = (8 * w + i) * 8 + lr;
    const int lc = swz(row, lane & 7);   // logical chunk stored in this lane's slot
    int64_t mr = m0 + row;
    if (mr > M - 1) mr = M - 1;
    ga[i] = A + mr * a.lda + lc * 8 - (i & 3) * 512;
    gb[i] = b_row<EPI, uint16_t>(a, n0 + row) + lc * 8 - (i & 3) * 512;
  }
}

template <int EPI, bool H>
__global__ __launch_bounds__(GT, 1) void k_gemm_bf16(GemmArgs a) {
  // two stages in distinct arrays: the compiler can then tell the in-flight
  // loads into one stage from the reads of the other and only waits at the
  // barrier that ends the stage
  __shared__ __attribute__((aligned(16))) uint16_t sA0[GM * GK];
  __shared__ __attribute__((aligned(16))) uint16_t sB0[GN * GK];
  __shared__ __attribute__((aligned(16))) uint16_t sA1[GM * GK];
  __shared__ __attribute__((aligned(16))) uint16_t sB1[GN * GK];
  __shared__ __attribute__((aligned(16))) float rbuf[GM];     // the tile's RMSNorm row scales
  __shared__ __attribute__((aligned(16))) int32_t pbuf[GM];   // the tile's token positions (QKV)
  __shared__ __attribute__((aligned(16))) float rvbuf[64];    // rotary frequencies of the lower-half dims (QKV)
  const int64_t M = *a.m_ptr;
  if (M <= 0) return;
  const int tiles_n = a.N / GN;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6, wm = w >> 1, wn = w & 1;
  const int nk = a.K / GK;   // even (the launcher checks K % 128)
  const uint16_t* A = static_cast<const uint16_t*>(a.A);

  // XCD-aware order: workgroups are dispatched round-robin over the 8 XCDs,
  // so workgroup b runs on XCD b % 8.  XCD x owns the M-tile rows
  // tm = x, x + 8, x + 16, ...; inside an XCD the tiles go in groups of
  // group_m of its rows, column by column, so the 32 workgroups resident on
  // one XCD share a few activation row-panels and a few weight column-panels
  // in that XCD's L2 instead of streaming 32 distinct panels.  Groups of 2
  // rows (gate/up 1-1.8 %, O 1-3.6 %, down 0.6-1.8 % faster than 4), 4 for
  // the q|k|v projection (2 is 2-3 % slower there).
  constexpr int group_m = EPI == EPI_QKV_ROPE ? 4 : 2;
  const int tiles_m = static_cast<int>((M + GM - 1) / GM);   // < 2^31 (M < 2^39)
  const int xcd = blockIdx.x & 7;
  const int per_xcd = gridDim.x >> 3;   // grid is a multiple of 8
  const int rows_x = tiles_m > xcd ? (tiles_m - xcd + 7) / 8 : 0;
  const int count_x = rows_x * tiles_n;
  const unsigned per_group = static_cast<unsigned>(group_m * tiles_n);
  auto tile_mn = [&](int q, int64_t& m0, int& n0) {
    const unsigned grp = static_cast<unsigned>(q) / per_group, within = static_cast<unsigned>(q) - grp * per_group;
    const int left = rows_x - static_cast<int>(grp) * group_m;
    const unsigned rows_here = left < group_m ? static_cast<unsigned>(left) : static_cast<unsigned>(group_m);   // 1 .. 4
    unsigned col, r;
    switch (rows_here) {   // within / rows_here without a division
      case 4: col = within >> 2; r = within & 3; break;
      case 2: col = within >> 1; r = within & 1; break;
      case 1: col = within; r = 0; break;
      default: col = within / 3; r = within - col * 3; break;
    }
    const int lr = static_cast<int>(grp) * group_m + static_cast<int>(r);
    m0 = static_cast<int64_t>(lr * 8 + xcd) * GM;
    n0 = static_cast<int>(col) * GN;
  };
  int q = blockIdx.x >> 3;
  if (q >= count_x) return;
  if (EPI == EPI_QKV_ROPE && t < (a.hd >> 1)) rvbuf[t] = a.rope_rev[t];   // visible after the first barrier
  const uint16_t* ga[8];
  const uint16_t* gb[8];
  int64_t m0;
  int n0;
  tile_mn(q, m0, n0);
  tile_sources<EPI>(a, A, M, m0, n0, w, lane, ga, gb);
  dma_stage(sA0, sB0, ga, gb, w);
  for (; q < count_x; q += per_xcd) {
    f32x16 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
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
    // nk is even: stages alternate 0, 1 and the loop has no odd tail (a
    // conditional second stage makes the compiler move the accumulators
    // between register files every iteration)
    for (int kt = 0; kt < nk; kt += 2) {
      mma_stage<H>(sA0, sB0, acc, wm, wn, lane, sA1, sB1, ga, gb, w, true);
      __syncthreads();
      mma_stage<H>(sA1, sB1, acc, wm, wn, lane, sA0, sB0, ga, gb, w, kt + 2 < nk);
      __syncthreads();
    }
    // stage 0 is free: the next tile's first k-step loads under the epilogue
    const bool more = q + per_xcd < count_x;
    int64_t m1 = 0;
    int n1 = 0;
    if (more) tile_mn(q + per_xcd, m1, n1);
    auto prefetch = [&]() {
      if (more) {
        tile_sources<EPI>(a, A, M, m1, n1, w, lane, ga, gb);
        dma_stage(sA0, sB0, ga, gb, w);
      }
    };
    // each wave stages its accumulators in its own 16 KB of stage 1, which is
    // idle until the next tile's first barrier
    float4* slice = reinterpret_cast<float4*>((w < 2 ? sA1 : sB1) + (w & 1) * 8192);
    epilogue_bf16<EPI, H>(a, acc, m0, n0, M, wm, wn, lane, slice, rbuf, pbuf, rvbuf, prefetch);
    m0 = m1;
    n0 = n1;
  }
  // the last tile's re-read of its last k-block lands before the workgroup
  // gives up its LDS
  __builtin_amdgcn_s_waitcnt(0);
}

hipError_t launch_gemm_bf16(int epi, const GemmArgs& a, hipStream_t s) {
  if (a.K <= 0 || a.K % (2 * GK) || a.N % GN) return hipErrorInvalidValue;   // whole pairs of k-steps, whole tiles
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
