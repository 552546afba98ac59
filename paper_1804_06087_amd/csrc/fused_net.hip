// Whole-network kernel for small image CNNs: one workgroup runs every layer of one
// model on one image, with the activations in LDS.
//
// For CIFAR-sized residual networks (ResNet-20: 16/32/64 channels at 32x32/16x16/8x8)
// each layer is a GEMM of a few MFLOPs per image: launched layer by layer over a batch,
// every launch is bound by its own load -> MFMA -> store latency and by the launch
// chain, not by arithmetic.  Here a workgroup keeps its image's tensors (at most a few
// tens of KB) in an LDS arena planned by liveness on the host, keeps the model's folded
// batch-norm scale / shift in LDS too, streams the weights (a copy in fragment order)
// from L2 through a register ring, and runs the layer program of its model:
// convolutions with folded batch-norm, residual and ReLU, the global average pool, and
// the final FC into the logits.
// Grid: x = image, y = the y-th selected model.
//
// Every value is bitwise the one the layer-by-layer path computes:
// * each output sums its K terms in the same (tap, channel) order, in the same 16-wide
//   groups, with the same v_mfma_f32_32x32x16_bf16 and the same operand roles
//   (weights as A, pixels as B) and positions (output channel co at row co % 32, GEMM
//   row m at column m % 32; an image's pixel p is row n * Ho * Wo + p of its layer,
//   with Ho * Wo a multiple of 32, so its column is p % 32; the FC's row is the image
//   index n); groups past K hold only zero products and are not run;
// * the epilogue is fma(acc, scale, shift), + residual, ReLU, one round to nearest
//   even bf16 (v_cvt_pk_bf16_f32 rounds as the integer form of the layer kernels does,
//   and the integer-max ReLU equals their fmaxf, for every finite value);
// * the average pool sums in the order of the batched kernel chosen for this batch
//   size (positions in sequence, or strided partial sums folded in order), then
//   multiplies by 1 / HW;
// * the FC logits are fma(acc, scale, shift) + 0.
#include "kernels.h"

namespace rafiki {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef const __attribute__((address_space(1))) bf16x8 gbf16x8;

__device__ __forceinline__ float fbf2f(uint32_t b16) { return __uint_as_float(b16 << 16); }
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {   // nearest even, a in the low half
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{a, b}, bf16x2));
}

constexpr int kRing = 8;                      // weight fragments in flight per lane
constexpr int kZeroOff = kFusedLdsBytes;      // 128 zero bytes after the arena: the padding reads

// LDS tensor layout: pixel p's row of Cs channels is R = Cs / 8 chunks of 16 bytes;
// logical chunk c sits in slot c ^ ((p >> (4 - log2 R)) & (R - 1)).  Sixteen lanes
// reading one chunk of 16 consecutive pixels (a B-operand fragment read) then touch
// 16 distinct 16-byte bank groups.
__device__ __forceinline__ int swz(int p, int Cs) {
  const int lr = 28 - __builtin_clz(Cs);   // log2(Cs / 8)
  return (int)__builtin_amdgcn_ubfe((unsigned)p, 4 - lr, lr);
}
__device__ __forceinline__ int chunk_addr(int base, int p, int c, int Cs) {
  return base + p * (Cs << 1) + ((c ^ swz(p, Cs)) << 4);
}

// One wave: output channels cb * 32 .. +31 of pixel blocks pb0 .. pb0 + CH - 1 of a
// KH x KH convolution over Cs = 16 * CPT input channels (CPT = 0: Cs = 8), input and
// output in LDS.  K group g (16 terms) is tap g / CPT, chunks 2 (g % CPT) + fk; with
// Cs = 8 lane half fk takes tap 2 g + fk.  The LDS address of every (block, tap) is
// computed once, with the swizzle folded in (a padding tap points at the zero chunk);
// a group then costs one XOR per block.
template <int CH, int KH, int CPT>
__device__ __forceinline__ void conv_chunk(const FusedLayer& L, char* lds, int cb, int pb0, int lane) {
  constexpr int TAPS = KH * KH;
  constexpr int NG = CPT > 0 ? TAPS * CPT : (TAPS + 1) / 2;
  constexpr int NQ = CPT > 0 ? TAPS : 2 * NG;   // Cs = 8: one past the last tap when TAPS is odd
  const int frow = lane & 31, fk = lane >> 5;
  gbf16x8* wrow = (gbf16x8*)L.w + ((size_t)cb * NG * 64 + lane);   // fragment order: group g at + 64 g
  bf16x8 ring[kRing];
#pragma unroll
  for (int i = 0; i < kRing; ++i)
    if (i < NG) ring[i] = wrow[64 * i];

  // q[j][t]: LDS byte address of tap t's first chunk for pixel block j (swizzle slot
  // folded in, this lane's half XORed in when Cs >= 16)
  const int R16 = L.Cs << 1;
  const int lr = 28 - __builtin_clz(L.Cs), sh = 4 - lr;
  const int fx = CPT > 0 ? fk : 0;
  int q[CH][NQ];
  if ((L.Wo & 31) == 0 && (L.W & 15) == 0) {
    // Each pixel block lies in one output row (wave-uniform ho), and the swizzle slot
    // of an input pixel depends on its column alone (W % 16 == 0): a tap's address is
    // a uniform row offset plus one of KH per-lane column parts.
#pragma unroll
    for (int j = 0; j < CH; ++j) {
      const int m0 = (pb0 + j) * 32;
      const int ho = m0 >> L.lwo;
      const int wi0 = ((m0 & (L.Wo - 1)) + frow) * L.stride - L.pad;
      int cpart[KH];
      bool cok[KH];
#pragma unroll
      for (int v = 0; v < KH; ++v) {
        const int wi = wi0 + v;
        cok[v] = (unsigned)wi < (unsigned)L.W;
        cpart[v] = L.in_off + wi * R16 + (((int)__builtin_amdgcn_ubfe((unsigned)wi, sh, lr) ^ fx) << 4);
      }
#pragma unroll
      for (int t = 0; t < NQ; ++t) {
        const int u = t / KH, v = t % KH;
        const int hi = ho * L.stride - L.pad + u;
        const bool rowok = t < TAPS && (unsigned)hi < (unsigned)L.H;   // wave-uniform
        q[j][t] = rowok && cok[v] ? cpart[v] + hi * L.W * R16 : kZeroOff;
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < CH; ++j) {
      const int p = (pb0 + j) * 32 + frow;
      const int ho = p >> L.lwo, wo = p & (L.Wo - 1);
      const int hi0 = ho * L.stride - L.pad, wi0 = wo * L.stride - L.pad;
      const int pin0 = hi0 * L.W + wi0;
#pragma unroll
      for (int t = 0; t < NQ; ++t) {
        const int u = t / KH, v = t % KH;
        const int pin = pin0 + u * L.W + v;
        const int a = L.in_off + pin * R16 + (((int)__builtin_amdgcn_ubfe((unsigned)pin, sh, lr) ^ fx) << 4);
        const bool ok = t < TAPS && (unsigned)(hi0 + u) < (unsigned)L.H && (unsigned)(wi0 + v) < (unsigned)L.W;
        q[j][t] = ok ? a : kZeroOff;
      }
    }
  }
  f32x16 acc[CH];
#pragma unroll
  for (int j = 0; j < CH; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[j][e] = 0.f;

  auto bread = [&](int g, bf16x8* b) {
#pragma unroll
    for (int j = 0; j < CH; ++j) {
      int a;
      if constexpr (CPT > 0) a = q[j][g / CPT] ^ ((2 * (g % CPT)) << 4);
      else a = fk ? q[j][2 * g + 1] : q[j][2 * g];
      b[j] = *(const bf16x8*)(lds + a);
    }
  };
  // B fragments D groups ahead: the LDS latency spans D groups of CH MFMAs each
  constexpr int D = CH == 1 ? 4 : (CH == 2 ? 2 : 1);
  bf16x8 bb[D + 1][CH];
#pragma unroll
  for (int i = 0; i < D; ++i)
    if (i < NG) bread(i, bb[i]);
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const bf16x8 a = ring[g % kRing];
    if (g + kRing < NG) ring[g % kRing] = wrow[64 * (g + kRing)];
    if (g + D < NG) bread(g + D, bb[(g + D) % (D + 1)]);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < CH; ++j)
      acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bb[g % (D + 1)][j], acc[j], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
  }

  // Epilogue: lane (frow, fk) holds channels cb * 32 + 8 qq + 4 fk + r (qq, r < 4) of
  // pixel (pb0 + j) * 32 + frow: 8 bytes of logical chunk cb * 4 + qq of that pixel.
  // Every LDS read (scale / shift, residual) is issued before the first write: the
  // output may replace the residual in place, and each (pixel, channel) is read and
  // written by this lane alone.  ReLU as an integer max with 0 equals fmaxf(v, 0) for
  // every value but NaN (-0 and negative values give +0).
  const int R16o = L.Cso << 1, c4 = (L.c_write + 3) & ~3;
  constexpr int NQQ = 4;
  int ro[CH], sw[CH];
  f32x4 sc[NQQ], sf[NQQ];
  uint2 rv[NQQ][CH];
#pragma unroll
  for (int j = 0; j < CH; ++j) {
    const int p = (pb0 + j) * 32 + frow;
    ro[j] = p * R16o + 8 * fk;
    sw[j] = swz(p, L.Cso);
  }
#pragma unroll
  for (int qq = 0; qq < NQQ; ++qq) {
    const int c = cb * 32 + 8 * qq + 4 * fk;
    if (c >= L.c_write) continue;
    sc[qq] = *(const f32x4*)(lds + L.ss_off + 4 * c);
    sf[qq] = *(const f32x4*)(lds + L.ss_off + 4 * (c4 + c));
    if (L.res_off >= 0) {
#pragma unroll
      for (int j = 0; j < CH; ++j) rv[qq][j] = *(const uint2*)(lds + L.res_off + ro[j] + (((cb * 4 + qq) ^ sw[j]) << 4));
    }
  }
#pragma unroll
  for (int qq = 0; qq < NQQ; ++qq) {
    const int c = cb * 32 + 8 * qq + 4 * fk;
    if (c >= L.c_write) continue;
#pragma unroll
    for (int j = 0; j < CH; ++j) {
      float v[4] = {__builtin_fmaf(acc[j][4 * qq + 0], sc[qq][0], sf[qq][0]),
                    __builtin_fmaf(acc[j][4 * qq + 1], sc[qq][1], sf[qq][1]),
                    __builtin_fmaf(acc[j][4 * qq + 2], sc[qq][2], sf[qq][2]),
                    __builtin_fmaf(acc[j][4 * qq + 3], sc[qq][3], sf[qq][3])};
      if (L.res_off >= 0) {
        const uint2 r = rv[qq][j];
        v[0] += fbf2f(r.x & 0xFFFFu); v[1] += fbf2f(r.x >> 16);
        v[2] += fbf2f(r.y & 0xFFFFu); v[3] += fbf2f(r.y >> 16);
      }
      if (L.relu) {
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] = __int_as_float(max(__float_as_int(v[r]), 0));
      }
      *(uint2*)(lds + L.out_off + ro[j] + (((cb * 4 + qq) ^ sw[j]) << 4)) =
          make_uint2(pack_bf16(v[0], v[1]), pack_bf16(v[2], v[3]));
    }
  }
}

template <int CH>
__device__ __forceinline__ void conv_chunk_cs(const FusedLayer& L, char* lds, int cb, int pb0, int lane) {
  if (L.kh == 3) {
    switch (L.Cs) {
      case 8: conv_chunk<CH, 3, 0>(L, lds, cb, pb0, lane); break;
      case 16: conv_chunk<CH, 3, 1>(L, lds, cb, pb0, lane); break;
      case 32: conv_chunk<CH, 3, 2>(L, lds, cb, pb0, lane); break;
      default: conv_chunk<CH, 3, 4>(L, lds, cb, pb0, lane); break;
    }
  } else {
    switch (L.Cs) {
      case 8: conv_chunk<CH, 1, 0>(L, lds, cb, pb0, lane); break;
      case 16: conv_chunk<CH, 1, 1>(L, lds, cb, pb0, lane); break;
      case 32: conv_chunk<CH, 1, 2>(L, lds, cb, pb0, lane); break;
      default: conv_chunk<CH, 1, 4>(L, lds, cb, pb0, lane); break;
    }
  }
}

__device__ __forceinline__ void run_conv(const FusedLayer& L, char* lds, int wave, int lane) {
  const int chunks_per_cb = (L.n_pb + L.ch - 1) / L.ch;
  const int chunks = chunks_per_cb * L.n_cb;
  for (int t = wave; t < chunks; t += kFusedWaves) {
    const int cb = t / chunks_per_cb, pb0 = (t - cb * chunks_per_cb) * L.ch;
    if (L.ch == 4) conv_chunk_cs<4>(L, lds, cb, pb0, lane);
    else if (L.ch == 2) conv_chunk_cs<2>(L, lds, cb, pb0, lane);
    else conv_chunk_cs<1>(L, lds, cb, pb0, lane);
  }
}

// Global average pool of the LDS tensor into a bf16 vector (an unswizzled row), in the
// summation order of the batched kernel that a batch of `batch` images uses: with
// batch * Cs / 8 >= 16384 every position in sequence; otherwise P = 256 / min(Cs / 8,
// 64) strided partial sums (partial s: positions s, s + P, ..., each from 0), folded
// in order onto partial 0.  A thread sums one 16-byte chunk (8 channels) of its
// positions; the partial sums go through tmp_off.  All threads must call it.
__device__ __forceinline__ void run_gap(const FusedLayer& L, char* lds, int batch, int tid) {
  const int HW = L.H * L.W, G = L.Cs >> 3;
  auto add8 = [&](float* acc, int p, int chk) {
    const uint4 v = *(const uint4*)(lds + chunk_addr(L.in_off, p, chk, L.Cs));
    acc[0] = acc[0] + fbf2f(v.x & 0xFFFFu); acc[1] = acc[1] + fbf2f(v.x >> 16);
    acc[2] = acc[2] + fbf2f(v.y & 0xFFFFu); acc[3] = acc[3] + fbf2f(v.y >> 16);
    acc[4] = acc[4] + fbf2f(v.z & 0xFFFFu); acc[5] = acc[5] + fbf2f(v.z >> 16);
    acc[6] = acc[6] + fbf2f(v.w & 0xFFFFu); acc[7] = acc[7] + fbf2f(v.w >> 16);
  };
  const float inv = 1.0f / (float)HW;
  if ((long long)batch * G >= 16384) {
    if (tid < G) {
      float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      for (int p = 0; p < HW; ++p) add8(acc, p, tid);
      uint4 o;
      o.x = pack_bf16(acc[0] * inv, acc[1] * inv); o.y = pack_bf16(acc[2] * inv, acc[3] * inv);
      o.z = pack_bf16(acc[4] * inv, acc[5] * inv); o.w = pack_bf16(acc[6] * inv, acc[7] * inv);
      *(uint4*)(lds + L.out_off + 16 * tid) = o;
    }
    return;
  }
  const int P = 256 / (G < 64 ? G : 64);
  float* part = (float*)(lds + L.tmp_off);   // [P][Cs]
  for (int i = tid; i < P * G; i += kFusedWaves * 64) {
    const int s = i / G, chk = i - s * G;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int p = s; p < HW; p += P) add8(acc, p, chk);
    float4* dst = (float4*)(part + s * L.Cs + 8 * chk);
    dst[0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
    dst[1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
  }
  __syncthreads();
  if (tid < L.Cs) {
    float acc = part[tid];
    for (int t = 1; t < P; ++t) acc = acc + part[t * L.Cs + tid];
    *(bf16_t*)(lds + L.out_off + 2 * tid) = (bf16_t)(pack_bf16(acc * inv, 0.f) & 0xFFFFu);
  }
}

// The final FC: logits of image n, its vector in column n % 32 of the B operand.
__device__ __forceinline__ void run_fc(const FusedLayer& L, const char* lds, int n, float* logits, int wave,
                                       int lane) {
  const int cb = wave;
  if (cb >= L.n_cb) return;
  const int frow = lane & 31, fk = lane >> 5;
  const bool mine = frow == (n & 31);
  f32x16 acc;
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[e] = 0.f;
  const int G = (L.K + 15) >> 4;
  gbf16x8* wrow = (gbf16x8*)L.w + ((size_t)cb * G * 64 + lane);
  for (int g = 0; g < G; ++g) {
    const int kk = g * 16 + 8 * fk;
    const bf16x8 a = wrow[64 * g];
    bf16x8 b = bf16x8{};
    if (mine && kk < L.K) b = *(const bf16x8*)(lds + L.in_off + 2 * kk);
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
  }
  if (!mine) return;
  const int c4 = (L.c_write + 3) & ~3;
  const float* sc = (const float*)(lds + L.ss_off);
#pragma unroll
  for (int q = 0; q < 4; ++q)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int c = cb * 32 + 8 * q + 4 * fk + r;
      if (c < L.c_write) logits[(long long)n * L.Cso + c] = __builtin_fmaf(acc[4 * q + r], sc[c], sc[c4 + c]) + 0.f;
    }
}

__global__ __launch_bounds__(kFusedWaves * 64, 2) void fused_net_kernel(FusedNetArgs a) {
  // the arena, the zero chunk of padding reads, the scale / shift table
  __shared__ uint4 lds4[(kFusedLdsBytes + 128 + kFusedTableBytes) / 16];
  char* lds = (char*)lds4;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = blockIdx.x, batch = gridDim.x;
  if (tid < 8) lds4[kZeroOff / 16 + tid] = make_uint4(0u, 0u, 0u, 0u);
  // the model of this workgroup: the blockIdx.y-th set bit of the mask
  unsigned m = a.mask;
  for (unsigned k = blockIdx.y; k > 0; --k) m &= m - 1;
  const int model = __builtin_ctz(m);
  const FusedLayer* prog = a.progs + (size_t)model * kFusedMaxLayers;
  float* logits = a.logits + (size_t)model * a.ld_model;
  FusedLayer L = prog[0];
  for (int li = 0; li + 1 < kFusedMaxLayers; ++li) {
    if (L.op == F_END) break;
    if (L.op == F_INPUT) {
      // the staged image, [pixel][Cso] rows -> the swizzled layout; the scale / shift table
      const int R = L.Cso >> 3, total = L.Ho * L.Wo * R;
      const uint4* src = (const uint4*)(a.in + (size_t)n * L.Ho * L.Wo * L.Cso);
      for (int i = tid; i < total; i += kFusedWaves * 64) {
        const int p = i / R, c = i - p * R;
        *(uint4*)(lds + chunk_addr(L.out_off, p, c, L.Cso)) = src[i];
      }
      const uint4* tab = (const uint4*)L.scale;
      for (int i = tid; i < (L.c_write >> 4); i += kFusedWaves * 64) lds4[L.ss_off / 16 + i] = tab[i];
    } else if (L.op == F_CONV) {
      run_conv(L, lds, wave, lane);
    } else if (L.op == F_GAP) {
      run_gap(L, lds, batch, tid);
    } else {
      run_fc(L, lds, n, logits, wave, lane);
    }
    __syncthreads();
    L = prog[li + 1];
  }
}

}  // namespace

hipError_t launch_fused_net(const FusedNetArgs& a, int n, int n_models, hipStream_t s) {
  if (n < 1 || n_models < 1 || n_models > 32 || __builtin_popcount(a.mask) != n_models) return hipErrorInvalidValue;
  launch(fused_net_kernel, dim3((unsigned)n, (unsigned)n_models), dim3(kFusedWaves * 64), s, a);
  return hipGetLastError();
}

}  // namespace rafiki
