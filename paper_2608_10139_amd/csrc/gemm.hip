// Dense projections of the prefill: C[M, N] = A[M, K] . W[N, K]^T with fused
// epilogues (rotary embedding on q/k, SwiGLU, GELU, residual add).
//
// bf16 path (gfx950 MFMA): 256 x 256 output tile per 512-thread workgroup,
// K stepped by 64 through a double-buffered LDS stage (2 x 64 KB).  Eight
// waves in a 2 x 4 grid each own a 128 x 64 sub-tile = 8 x 4 blocks of
// v_mfma_f32_16x16x32_bf16.  The weight block is the MFMA's first operand and
// the activation block its second, so every lane ends up holding four
// consecutive output columns of one row: stores are 8- or 16-byte vectors and
// the column pairs the epilogues need (rotary halves, gate/up) sit in the
// same lane.  LDS rows are 128 bytes; the 16-byte chunk index is XORed with
// (row & 7) so the 16 rows a fragment read touches fall in distinct banks.
//
// M (tokens in the chunk) is read from device memory; the grid is persistent
// (one workgroup per CU) and walks the tiles, so an empty chunk costs one
// launch and no work.
//
// fp32 path: a plain 64 x 64 LDS-tiled FMA kernel with the same row mapping
// and epilogues, used for fp32 models.
#include "aiq_internal.h"

namespace aiq {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

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

__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
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
    // interleave 16-row groups: gate rows 16b.., up rows 16b.., ...
    const int b16 = n >> 4, r = n & 15;
    const int row = (b16 >> 1) * 16 + r;
    return static_cast<const T*>((b16 & 1) ? a.B1 : a.B0) + static_cast<int64_t>(row) * a.K;
  } else {
    return static_cast<const T*>(a.B0) + static_cast<int64_t>(n) * a.K;
  }
}

// ======================================================================= bf16 MFMA
constexpr int GM = 256, GN = 256, GK = 64, GT = 512;
constexpr int STAGE = (GM + GN) * GK;   // bf16 elements per LDS stage

template <int EPI>
__device__ __forceinline__ void epilogue_bf16(const GemmArgs& a, f32x4 (&acc)[4][8], int64_t m0, int n0,
                                              int64_t M, int wm, int wn, int lane) {
  const int c4 = 4 * (lane >> 4);
  const int nw = n0 + wn * 64;   // first GEMM column of this wave
#pragma unroll
  for (int mi = 0; mi < 8; ++mi) {
    const int64_t m = m0 + wm * 128 + mi * 16 + (lane & 15);
    if (m >= M) continue;
    if (EPI == EPI_STORE_F32) {
      float* C = static_cast<float*>(a.C) + m * a.ldc;
#pragma unroll
      for (int ni = 0; ni < 4; ++ni) {
        const f32x4 v = acc[ni][mi];
        *reinterpret_cast<float4*>(C + nw + ni * 16 + c4) = make_float4(v[0], v[1], v[2], v[3]);
      }
    } else if (EPI == EPI_STORE_ACT) {
      uint16_t* C = static_cast<uint16_t*>(a.C) + m * a.ldc;
#pragma unroll
      for (int ni = 0; ni < 4; ++ni) {
        const f32x4 v = acc[ni][mi];
        *reinterpret_cast<uint2*>(C + nw + ni * 16 + c4) = pack_bf16x4(v[0], v[1], v[2], v[3]);
      }
    } else if (EPI == EPI_RESID) {
      float* X = a.X + m * a.ldx;
#pragma unroll
      for (int ni = 0; ni < 4; ++ni) {
        float4* px = reinterpret_cast<float4*>(X + nw + ni * 16 + c4);
        float4 x = *px;
        const f32x4 v = acc[ni][mi];
        x.x += v[0]; x.y += v[1]; x.z += v[2]; x.w += v[3];
        *px = x;
      }
    } else if (EPI == EPI_SWIGLU) {
      uint16_t* C = static_cast<uint16_t*>(a.C) + m * a.ldc;
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        const f32x4 g = acc[2 * p][mi], u = acc[2 * p + 1][mi];
        const int col = nw / 2 + p * 16 + c4;
        *reinterpret_cast<uint2*>(C + col) =
            pack_bf16x4(silu(g[0]) * u[0], silu(g[1]) * u[1], silu(g[2]) * u[2], silu(g[3]) * u[3]);
      }
    } else if (EPI == EPI_QKV_ROPE) {
      uint16_t* C = static_cast<uint16_t*>(a.C) + m * a.ldc;
      if (nw >= a.n_q + a.n_kv) {  // v: stored as is
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) {
          const f32x4 v = acc[ni][mi];
          *reinterpret_cast<uint2*>(C + nw + ni * 16 + c4) = pack_bf16x4(v[0], v[1], v[2], v[3]);
        }
      } else {
        const int sbase = nw < a.n_q ? 0 : a.n_q;
        const int c = nw - sbase;
        const int head = c / a.hd;
        const int hh = (c % a.hd) >> 6;   // 0 except the second half-wave of a 128-dim head
        const int half = a.hd >> 1;
        const int p = a.pos[m];
        const float* cs = a.rope_cos + static_cast<int64_t>(p) * half;
        const float* sn = a.rope_sin + static_cast<int64_t>(p) * half;
        uint16_t* Ch = C + sbase + head * a.hd;
#pragma unroll
        for (int ni = 0; ni < 2; ++ni) {
          const int dlo = hh * 32 + ni * 16 + c4;   // lower-half dim of this lane's 4 columns
          const f32x4 x1 = acc[ni][mi], x2 = acc[ni + 2][mi];
          const float4 cv = *reinterpret_cast<const float4*>(cs + dlo);
          const float4 sv = *reinterpret_cast<const float4*>(sn + dlo);
          *reinterpret_cast<uint2*>(Ch + dlo) =
              pack_bf16x4(x1[0] * cv.x - x2[0] * sv.x, x1[1] * cv.y - x2[1] * sv.y,
                          x1[2] * cv.z - x2[2] * sv.z, x1[3] * cv.w - x2[3] * sv.w);
          *reinterpret_cast<uint2*>(Ch + dlo + half) =
              pack_bf16x4(x2[0] * cv.x + x1[0] * sv.x, x2[1] * cv.y + x1[1] * sv.y,
                          x2[2] * cv.z + x1[2] * sv.z, x2[3] * cv.w + x1[3] * sv.w);
        }
      }
    }
  }
}

template <int EPI>
__global__ __launch_bounds__(GT) void k_gemm_bf16(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[2 * STAGE];
  const int64_t M = *a.m_ptr;
  if (M <= 0) return;
  const int tiles_n = a.N / GN;
  const int64_t n_tiles = ((M + GM - 1) / GM) * tiles_n;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6, wm = w >> 2, wn = w & 3;
  const int nk = a.K / GK;
  const uint16_t* A = static_cast<const uint16_t*>(a.A);

  for (int64_t tile = blockIdx.x; tile < n_tiles; tile += gridDim.x) {
    const int64_t m0 = (tile / tiles_n) * GM;
    const int n0 = static_cast<int>(tile % tiles_n) * GN;
    const uint16_t* ap[4];
    const uint16_t* bp[4];
    int so[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int id = i * GT + t, row = id >> 3, ch = id & 7;
      int64_t mr = m0 + row;
      if (mr > M - 1) mr = M - 1;
      ap[i] = A + mr * a.lda + ch * 8;
      bp[i] = b_row<EPI, uint16_t>(a, n0 + row) + ch * 8;
      so[i] = row * GK + ((ch ^ (row & 7)) << 3);
    }
    uint4 ra[4], rb[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ra[i] = *reinterpret_cast<const uint4*>(ap[i]);
      rb[i] = *reinterpret_cast<const uint4*>(bp[i]);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      *reinterpret_cast<uint4*>(lds + so[i]) = ra[i];
      *reinterpret_cast<uint4*>(lds + GM * GK + so[i]) = rb[i];
    }
    __syncthreads();

    f32x4 acc[4][8];
#pragma unroll
    for (int ni = 0; ni < 4; ++ni)
#pragma unroll
      for (int mi = 0; mi < 8; ++mi) acc[ni][mi] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int kt = 0; kt < nk; ++kt) {
      const int st = kt & 1;
      const uint16_t* As = lds + st * STAGE;
      const uint16_t* Bs = As + GM * GK;
      const bool more = kt + 1 < nk;
      if (more) {
        const int ko = (kt + 1) * GK;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          ra[i] = *reinterpret_cast<const uint4*>(ap[i] + ko);
          rb[i] = *reinterpret_cast<const uint4*>(bp[i] + ko);
        }
      }
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const int ch = kk * 4 + (lane >> 4);
        const int sw = (ch ^ (lane & 7)) << 3;   // row & 7 == lane & 7 for every fragment row
        bf16x8 af[8], bw[4];
#pragma unroll
        for (int mi = 0; mi < 8; ++mi)
          af[mi] = *reinterpret_cast<const bf16x8*>(As + (wm * 128 + mi * 16 + (lane & 15)) * GK + sw);
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
          bw[ni] = *reinterpret_cast<const bf16x8*>(Bs + (wn * 64 + ni * 16 + (lane & 15)) * GK + sw);
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
#pragma unroll
          for (int mi = 0; mi < 8; ++mi)
            acc[ni][mi] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bw[ni], af[mi], acc[ni][mi], 0, 0, 0);
      }
      if (more) {
        uint16_t* As2 = lds + (st ^ 1) * STAGE;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          *reinterpret_cast<uint4*>(As2 + so[i]) = ra[i];
          *reinterpret_cast<uint4*>(As2 + GM * GK + so[i]) = rb[i];
        }
      }
      __syncthreads();
    }
    epilogue_bf16<EPI>(a, acc, m0, n0, M, wm, wn, lane);
  }
}

hipError_t launch_gemm_bf16(int epi, const GemmArgs& a, hipStream_t s) {
  const int64_t tiles = ((a.m_ub + GM - 1) / GM) * (a.N / GN);
  int64_t g = num_cus();
  if (tiles < g) g = tiles;
  if (g < 1) g = 1;
  const dim3 grid(static_cast<unsigned>(g)), block(GT);
  switch (epi) {
    case EPI_STORE_F32: hipLaunchKernelGGL(k_gemm_bf16<EPI_STORE_F32>, grid, block, 0, s, a); break;
    case EPI_STORE_ACT: hipLaunchKernelGGL(k_gemm_bf16<EPI_STORE_ACT>, grid, block, 0, s, a); break;
    case EPI_RESID: hipLaunchKernelGGL(k_gemm_bf16<EPI_RESID>, grid, block, 0, s, a); break;
    case EPI_SWIGLU: hipLaunchKernelGGL(k_gemm_bf16<EPI_SWIGLU>, grid, block, 0, s, a); break;
    case EPI_QKV_ROPE: hipLaunchKernelGGL(k_gemm_bf16<EPI_QKV_ROPE>, grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
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
      if (EPI == EPI_RESID) {
        float4* px = reinterpret_cast<float4*>(a.X + m * a.ldx + n);
        float4 x = *px;
        x.x += acc[i][0]; x.y += acc[i][1]; x.z += acc[i][2]; x.w += acc[i][3];
        *px = x;
      } else if (EPI == EPI_GELU) {
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
    case EPI_RESID: hipLaunchKernelGGL(k_gemm_f32<EPI_RESID>, grid, block, 0, s, a); break;
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
