// bf16 implicit-GEMM convolution / FC on gfx950 matrix cores.
//
// GEMM view: out[m, co] = sum_k X[m, k] * Wp[co, k], with m an output pixel
// (n, ho, wo), co an output channel and k = (u, v, ci) a kernel tap and input
// channel.  X is never materialised: each 16-byte chunk of a tile row is 8
// consecutive input channels of one tap, loaded straight from the NHWC tensor
// (zero outside the image or past K).  Weights are pre-packed [Co_pad][Kp] with K in
// the same (u, v, ci) order, so a weight tile row is a contiguous 128-byte run.
//
// Block tile BM pixels x BN channels x 64 K, staged through LDS (double buffered,
// 16-byte chunks XOR-swizzled by row so the per-lane fragment reads are
// bank-conflict free).  Each wave owns a (BM/WM) x (BN/WN) sub-tile computed with
// v_mfma_f32_32x32x16_bf16: the weight fragment is the MFMA "A" operand (rows =
// channels) and the pixel fragment the "B" operand (columns = pixels), so each lane
// ends with 4 runs of 4 consecutive channels of one pixel -- 8-byte NHWC stores.
//
// Epilogue (fused): y = acc * scale[co] + shift[co] (+ residual), ReLU, round to
// bf16 (nearest even) or keep fp32; or raw fp32 partial sums for split-K.
#include "kernels.h"

namespace rafiki {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float bf2f(uint32_t b16) { return __uint_as_float(b16 << 16); }

// fp32 -> bf16 bits, round to nearest, ties to even (finite inputs).
__device__ __forceinline__ uint32_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

template <int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(WM * WN * 64) void conv_bf16_kernel(ConvArgs a) {
  constexpr int NT = WM * WN * 64;
  constexpr int BK = 64;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int RPP = NT / 8;          // tile rows covered per load pass (8 chunks per row)
  constexpr int AP = BM / RPP, BP = BN / RPP;
  static_assert(TM >= 1 && TN >= 1 && AP >= 1 && BP >= 1, "tile shape");

  __shared__ uint4 lds[2][(BM + BN) * 8];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave % WM, wn = wave / WM;
  const int nt = blockIdx.x % a.n_tiles, mt = blockIdx.x / a.n_tiles;
  const int m0 = mt * BM, n0 = nt * BN;
  const int ktiles = a.Kp / BK;
  const int kt_begin = blockIdx.y * a.kt_per_split;
  const int nk = min(a.kt_per_split, ktiles - kt_begin);

  const bf16_t* __restrict__ X = (const bf16_t*)a.x;
  const bf16_t* __restrict__ Wt = (const bf16_t*)a.w;
  const int chunk = tid & 7;
  const int rbase = tid >> 3;

  // Per-row input geometry of the pixels this thread loads.
  long long a_img[AP];
  int a_hi[AP], a_wi[AP];
  const int HoWo = a.Ho * a.Wo;
#pragma unroll
  for (int p = 0; p < AP; ++p) {
    const int m = m0 + rbase + p * RPP;
    if (m < a.M) {
      const int n = m / HoWo, r = m - n * HoWo;
      const int ho = r / a.Wo, wo = r - ho * a.Wo;
      a_img[p] = (long long)n * a.H * a.W * a.Cs;
      a_hi[p] = ho * a.stride - a.pad;
      a_wi[p] = wo * a.stride - a.pad;
    } else {
      a_img[p] = 0;
      a_hi[p] = -(1 << 28);   // never inside the image
      a_wi[p] = 0;
    }
  }

  uint4 ra[AP], rb[BP];
  auto gload = [&](int kt) {
    const int k = (kt_begin + kt) * BK + chunk * 8;
    const int tap = k / a.Cs;
    const int ci = k - tap * a.Cs;
    const int u = tap / a.kw, v = tap - u * a.kw;
    const bool kvalid = k < a.K;
#pragma unroll
    for (int p = 0; p < AP; ++p) {
      const int hi = a_hi[p] + u, wi = a_wi[p] + v;
      if (kvalid && (unsigned)hi < (unsigned)a.H && (unsigned)wi < (unsigned)a.W) {
        ra[p] = *(const uint4*)(X + a_img[p] + ((long long)hi * a.W + wi) * a.Cs + ci);
      } else {
        ra[p] = make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int p = 0; p < BP; ++p) {
      const int row = rbase + p * RPP;
      rb[p] = *(const uint4*)(Wt + (long long)(n0 + row) * a.Kp + k);
    }
  };
  auto sstore = [&](int buf) {
    uint4* As = lds[buf];
    uint4* Bs = lds[buf] + BM * 8;
#pragma unroll
    for (int p = 0; p < AP; ++p) {
      const int row = rbase + p * RPP;
      As[row * 8 + (chunk ^ (row & 7))] = ra[p];
    }
#pragma unroll
    for (int p = 0; p < BP; ++p) {
      const int row = rbase + p * RPP;
      Bs[row * 8 + (chunk ^ (row & 7))] = rb[p];
    }
  };

  f32x16 acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  if (nk > 0) {
    gload(0);
    sstore(0);
  }
  __syncthreads();

  const int frow = lane & 31, fk = lane >> 5;
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
    const uint4* As = lds[cur];
    const uint4* Bs = lds[cur] + BM * 8;
#pragma unroll
    for (int s = 0; s < BK / 16; ++s) {
      const int kc = 2 * s + fk;
      bf16x8 xf[TM], wf[TN];
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) {
        const int r = wm * WTM + tm * 32 + frow;
        uint4 q = As[r * 8 + (kc ^ (r & 7))];
        xf[tm] = __builtin_bit_cast(bf16x8, q);
      }
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        const int r = wn * WTN + tn * 32 + frow;
        uint4 q = Bs[r * 8 + (kc ^ (r & 7))];
        wf[tn] = __builtin_bit_cast(bf16x8, q);
      }
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
          acc[tn][tm] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[tn], xf[tm], acc[tn][tm], 0, 0, 0);
    }
    if (kt + 1 < nk) sstore(cur ^ 1);
    __syncthreads();
  }

  // ---- epilogue: lane holds channels n0 + wn*WTN + tn*32 + 8g + 4*fk + j of pixel
  //      m0 + wm*WTM + tm*32 + frow, for g, j in 0..3.
  const bool split = gridDim.y > 1;
#pragma unroll
  for (int tn = 0; tn < TN; ++tn) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int c = n0 + wn * WTN + tn * 32 + 8 * g + 4 * fk;
      if (split) {
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) {
          const int m = m0 + wm * WTM + tm * 32 + frow;
          if (m < a.M) {
            float4 v = make_float4(acc[tn][tm][4 * g + 0], acc[tn][tm][4 * g + 1], acc[tn][tm][4 * g + 2],
                                   acc[tn][tm][4 * g + 3]);
            *(float4*)(a.partial + ((long long)blockIdx.y * a.M + m) * a.Co_pad + c) = v;
          }
        }
        continue;
      }
      if (c >= a.c_write) continue;
      const float4 sc = *(const float4*)(a.scale + c);
      const float4 sh = *(const float4*)(a.shift + c);
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) {
        const int m = m0 + wm * WTM + tm * 32 + frow;
        if (m >= a.M) continue;
        float v0 = acc[tn][tm][4 * g + 0] * sc.x + sh.x;
        float v1 = acc[tn][tm][4 * g + 1] * sc.y + sh.y;
        float v2 = acc[tn][tm][4 * g + 2] * sc.z + sh.z;
        float v3 = acc[tn][tm][4 * g + 3] * sc.w + sh.w;
        const long long o = (long long)m * a.ldy + c;
        if (a.res) {
          const uint2 r = *(const uint2*)((const bf16_t*)a.res + o);
          v0 += bf2f(r.x & 0xFFFFu);
          v1 += bf2f(r.x >> 16);
          v2 += bf2f(r.y & 0xFFFFu);
          v3 += bf2f(r.y >> 16);
        }
        if (a.relu) {
          v0 = fmaxf(v0, 0.f); v1 = fmaxf(v1, 0.f); v2 = fmaxf(v2, 0.f); v3 = fmaxf(v3, 0.f);
        }
        if (a.out_f32) {
          float* y = (float*)a.y + o;
          y[0] = v0;
          if (c + 1 < a.c_write) y[1] = v1;
          if (c + 2 < a.c_write) y[2] = v2;
          if (c + 3 < a.c_write) y[3] = v3;
        } else {
          uint2 q;
          q.x = f2bf(v0) | (f2bf(v1) << 16);
          q.y = f2bf(v2) | (f2bf(v3) << 16);
          *(uint2*)((bf16_t*)a.y + o) = q;
        }
      }
    }
  }
}

// Sum the split-K partials in split order, then the same epilogue as above.
// One thread per (row, 4-channel group).
__global__ void splitk_reduce_kernel(ConvArgs a, int splits, int in_bf16) {
  const int groups = (a.c_write + 3) / 4;
  const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long long)a.M * groups) return;
  const int m = (int)(idx / groups);
  const int c = (int)(idx - (long long)m * groups) * 4;
  float4 s = *(const float4*)(a.partial + (long long)m * a.Co_pad + c);
  for (int z = 1; z < splits; ++z) {
    const float4 t = *(const float4*)(a.partial + ((long long)z * a.M + m) * a.Co_pad + c);
    s.x += t.x; s.y += t.y; s.z += t.z; s.w += t.w;
  }
  const float4 sc = *(const float4*)(a.scale + c);
  const float4 sh = *(const float4*)(a.shift + c);
  float v[4] = {s.x * sc.x + sh.x, s.y * sc.y + sh.y, s.z * sc.z + sh.z, s.w * sc.w + sh.w};
  const long long o = (long long)m * a.ldy + c;
  if (a.res) {
    for (int j = 0; j < 4; ++j) {
      if (c + j >= a.c_write) break;
      if (in_bf16) v[j] += bf2f(((const bf16_t*)a.res)[o + j]);
      else v[j] += ((const float*)a.res)[o + j];
    }
  }
  for (int j = 0; j < 4; ++j) {
    if (c + j >= a.c_write) break;
    float t = a.relu ? fmaxf(v[j], 0.f) : v[j];
    if (a.out_f32) ((float*)a.y)[o + j] = t;
    else ((bf16_t*)a.y)[o + j] = (bf16_t)f2bf(t);
  }
}

template <int BM, int BN, int WM, int WN>
static hipError_t launch_cfg(const ConvArgs& a, int splits, hipStream_t s) {
  ConvArgs b = a;
  b.n_tiles = (a.Co_pad + BN - 1) / BN;
  const int m_tiles = (a.M + BM - 1) / BM;
  dim3 grid(m_tiles * b.n_tiles, splits);
  hipLaunchKernelGGL((conv_bf16_kernel<BM, BN, WM, WN>), grid, dim3(WM * WN * 64), 0, s, b);
  return hipGetLastError();
}

hipError_t launch_conv_bf16(const ConvArgs& a, int bm, int bn, int splits, hipStream_t s) {
  if (bn == 128) {
    if (bm == 128) return launch_cfg<128, 128, 2, 2>(a, splits, s);
    if (bm == 64) return launch_cfg<64, 128, 1, 4>(a, splits, s);
    if (bm == 32) return launch_cfg<32, 128, 1, 4>(a, splits, s);
  } else if (bn == 64) {
    if (bm == 128) return launch_cfg<128, 64, 2, 2>(a, splits, s);
    if (bm == 64) return launch_cfg<64, 64, 2, 2>(a, splits, s);
    if (bm == 32) return launch_cfg<32, 64, 1, 2>(a, splits, s);
  } else if (bn == 32) {
    if (bm == 128) return launch_cfg<128, 32, 4, 1>(a, splits, s);
    if (bm == 64) return launch_cfg<64, 32, 2, 1>(a, splits, s);
    if (bm == 32) return launch_cfg<32, 32, 1, 1>(a, splits, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_splitk_reduce(const ConvArgs& a, int splits, int in_bf16, hipStream_t s) {
  const long long total = (long long)a.M * ((a.c_write + 3) / 4);
  const int threads = 256;
  const long long blocks = (total + threads - 1) / threads;
  hipLaunchKernelGGL(splitk_reduce_kernel, dim3((unsigned)blocks), dim3(threads), 0, s, a, splits, in_bf16);
  return hipGetLastError();
}

}  // namespace rafiki
