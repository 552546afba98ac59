// bf16 implicit-GEMM convolution / FC on gfx950 matrix cores, direct-to-LDS pipeline.
//
// GEMM view: out[m, co] = sum_k X[m, k] * Wp[co, k]; m = output pixel (n, ho, wo),
// co = output channel, k = (u, v, ci) kernel tap and input channel.  X is gathered
// on the fly from the NHWC input: a 16-byte chunk of a tile row is 8 consecutive
// channels of one tap.
//
// Tiles move HBM -> LDS with buffer_load_dwordx4 ... lds (no register staging).  A
// lane whose chunk lies outside the image or past K gets an offset beyond the
// buffer's num_records, for which the hardware writes zeros: that is the zero
// padding.  STAGES K tiles of 64 are in flight in an LDS ring, laid out with the
// bank-conflict-free swizzle described at swz<KC>().  Each wave computes a (BM/WM) x (BN/WN) sub-tile with
// v_mfma_f32_32x32x16_bf16 (weights = A operand, pixels = B operand), so a lane ends
// with runs of 4 consecutive channels of one pixel.  Fused epilogue: fp32 scale /
// shift (folded batch-norm + bias), residual, ReLU, bf16 store; or fp32 output;
// or raw fp32 split-K partials.
#include "kernels.h"

namespace rafiki {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ float bf2f_m(uint32_t b16) { return __uint_as_float(b16 << 16); }
__device__ __forceinline__ uint32_t f2bf_m(float f) {   // nearest, ties to even (finite)
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}
// Two values rounded to bf16 by v_cvt_pk_bf16_f32 (nearest even: the same bits as
// f2bf_m for every finite value), a in the low half.
typedef __bf16 bf16x2_m __attribute__((ext_vector_type(2)));
typedef float f32x2_m __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack2_bf16(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_m{a, b}, bf16x2_m));
}
// ReLU as an integer max with 0: the same bits as fmaxf(v, 0) for every value but NaN
// (negative values and -0 give +0, as fmaxf does on this hardware), in one instruction.
__device__ __forceinline__ float relu_m(float v) { return __int_as_float(max(__float_as_int(v), 0)); }

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// LDS tile layout: a K tile is 64 (KC = 8 chunks of 16 bytes per row) or 32 (KC = 4)
// channels wide; row r keeps logical chunk c in slot c ^ swz<KC>(r).  A 16-byte
// fragment read serves 16 lanes at a time across 64 four-byte banks; its 16 lanes
// read 16 consecutive rows of one chunk.
//   KC = 8: swz(r) = (r & 7) ^ ((r >> 3) & 1) keeps (r % 2, slot) distinct over any
//           16 rows (a 128-byte row spans half of the banks);
//   KC = 4: swz(r) = (r >> 2) & 3 keeps (r % 4, slot) distinct over 16 rows (a
//           64-byte row spans a quarter of the banks).
// Either way the reads are bank-conflict free.
template <int KC>
__device__ __forceinline__ int swz(int r) {
  return KC == 8 ? ((r & 7) ^ ((r >> 3) & 1)) : ((r >> 2) & 3);
}

// Per-thread state of the HBM -> LDS tile loader.  One load instruction moves 64
// chunks = ROWS = 64 / KC tile rows.  Wave w's instruction j fills rows
// (j * NW + w) * ROWS .. +ROWS, lane l -> slot l % KC of row l / KC of the group.
//   KC = 8: with NW even that row's swz is (l / 8) ^ (w & 1) for every j, so lane l
//           always carries chunk (l % 8) ^ (l / 8) ^ (w & 1);
//   KC = 4: the group starts at a multiple of 16 rows, so the row's swz is l / 16 and
//           lane l always carries chunk (l % 4) ^ (l / 16).
//
// ALIGNED (Cs % 64 == 0): K is ordered (channel block of 64, tap, channel), so a
// 64-wide K block is channel block gk / taps at tap gk % taps (a 32-wide K tile is
// one half of such a block).  The taps of one channel block are consecutive tiles:
// they re-read the same input rows while those are still in L2.  Tap, channel block
// and half are wave-uniform and advanced incrementally; per row only the
// image-bounds test and one add remain.  A tile of fused conv1d branches runs only
// the first `taps` taps of each channel block; its weight K tile then follows the
// packed stride of tap_stride taps per block.  Otherwise (Cs % 64 != 0) K is ordered
// (tap, channel) and each lane decodes its own (u, v, ci) with multiply-high division.
template <int BM, int BN, int NW, bool ALIGNED, int KC, bool TL>
struct Loader {
  static constexpr int ROWS = 64 / KC;
  static constexpr int SUBS = 8 / KC;      // K tiles per 64-channel block
  static constexpr int RA = BM / (ROWS * NW);
  static constexpr int RB = BN / (ROWS * NW);
  static constexpr int STAGE_CHUNKS = (BM + BN) * KC;
  static_assert(KC == 8 || KC == 4, "K tile of 64 or 32 channels");
  __amdgpu_buffer_rsrc_t xr, wr;
  unsigned oob;
  int chunk, wave, kt_begin;
  int a_img[RA], a_hi[RA], a_wi[RA];   // general path: image base pixel, top-left input coords
  int a_off[RA];                       // aligned path: byte offset of (hi0, wi0, chunk) (may be virtual)
  unsigned b_off[RB];
  int nu, nv, ntap, ncb, nsub;         // aligned path: tap (u, v, index), channel block, half of the next tile
  int taps, tstride, cs;               // TL: taps run per channel block; taps packed per block; Cs
  // TL with token ids: the table rows under taps 0-3 (tk0) and 4-7 (tk1) of row j,
  // 16 bits each (0xFFFF: zeros).  Packed words selected by shifts keep them in
  // registers (an array indexed by the tap would be moved to scratch memory).
  uint64_t tk0[TL ? RA : 1], tk1[TL ? RA : 1];

  __device__ __forceinline__ void init(const ConvArgs& a, int m0, int n0, int wave_, int lane, int kt_begin_,
                                       int taps_) {
    wave = wave_;
    kt_begin = kt_begin_;
    taps = TL ? taps_ : a.kh * a.kw;
    tstride = TL ? a.tap_stride : 0;
    cs = a.Cs;
    const int lrow = lane / KC;
    chunk = KC == 8 ? ((lane & 7) ^ lrow ^ (wave & 1)) : ((lane & 3) ^ (lane >> 4));
    xr = __builtin_amdgcn_make_buffer_rsrc((void*)a.x, (short)0, a.x_bytes, 0x00020000);
    wr = __builtin_amdgcn_make_buffer_rsrc((void*)a.w, (short)0, a.w_bytes, 0x00020000);
    oob = (unsigned)a.x_bytes;   // offset at num_records: the hardware returns zeros
    const int HoWo = a.Ho * a.Wo;
#pragma unroll
    for (int j = 0; j < RA; ++j) {
      const int m = m0 + (j * NW + wave) * ROWS + lrow;
      if (m < a.M) {
        int n, ho, wo;
        if (a.pool2) {   // row m: position m % 4 of 2x2 window m / 4
          const int q = m >> 2, Wo2 = a.Wo >> 1, HW2 = (a.Ho >> 1) * Wo2;
          n = q / HW2;
          const int r = q - n * HW2, ho2 = r / Wo2;
          ho = 2 * ho2 + ((m >> 1) & 1);
          wo = 2 * (r - ho2 * Wo2) + (m & 1);
        } else {
          n = m / HoWo;
          const int r = m - n * HoWo;
          ho = r / a.Wo;
          wo = r - ho * a.Wo;
        }
        a_img[j] = n * a.H * a.W;
        a_hi[j] = ho * a.stride - a.pad;
        a_wi[j] = wo * a.stride - a.pad;
      } else {
        a_img[j] = 0;
        a_hi[j] = -(1 << 28);
        a_wi[j] = 0;
      }
      a_off[j] = ((a_img[j] + a_hi[j] * a.W + a_wi[j]) * a.Cs + chunk * 8) * 2;
      if constexpr (TL) {
        if (a.tok) {
          const int rows = a.x_bytes / (a.Cs * 2);   // table rows (< 0xFFFF)
          tk0[j] = 0;
          tk1[j] = 0;
#pragma unroll
          for (int v = 0; v < kMaxGatherTaps; ++v) {
            const int wi = a_wi[j] + v;
            int id = -1;
            if (a_hi[j] == 0 && v < a.kw && (unsigned)wi < (unsigned)a.W) id = a.tok[a_img[j] + wi];
            const uint64_t f = (unsigned)id < (unsigned)rows ? (uint64_t)id : 0xFFFFull;
            if (v < 4) tk0[j] |= f << (16 * v);
            else tk1[j] |= f << (16 * (v - 4));
          }
        }
      }
    }
#pragma unroll
    for (int j = 0; j < RB; ++j)
      b_off[j] = (unsigned)(((n0 + (j * NW + wave) * ROWS + lrow) * a.Kp + chunk * 8) * 2);
    if (ALIGNED) {
      const int blk = kt_begin / SUBS;
      nsub = kt_begin - blk * SUBS;
      ncb = blk / taps;
      ntap = blk - ncb * taps;
      nu = ntap / a.kw;
      nv = ntap - nu * a.kw;
    }
  }

  // Token gather (TL): the pixel rows of the next K tile come from the table rows of
  // their tokens under tap ntap, at channel block ncb.
  template <int P, int NP>
  __device__ __forceinline__ void issue_gather(uint4* sbase) {
    const int cdelta = (ncb * 64 + nsub * (8 * KC) + chunk * 8) * 2;
    const int sh = 16 * (ntap & 3);
#pragma unroll
    for (int j = P; j < RA; j += NP) {
      const uint64_t w = ntap < 4 ? tk0[j] : tk1[j];
      const unsigned id = (unsigned)(w >> sh) & 0xFFFFu;
      const unsigned off = id != 0xFFFFu ? id * (unsigned)(2 * cs) + (unsigned)cdelta : oob;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void*)(sbase + (j * NW + wave) * 64), 16, off, 0, 0, 0);
    }
    if (P == NP - 1 && ++nsub == SUBS) {
      nsub = 0;
      if (++ntap == taps) {
        ntap = 0;
        ++ncb;
      }
    }
  }

  // Issue the loads of K tile kt (relative to the split's first tile) into LDS stage
  // `stage`, or only part P of NP of them (the loads j with j % NP == P), so that a
  // tile's loads can be spread over the k-steps of the running tile.  The parts of a
  // tile are issued in order, and tiles in increasing kt order (the aligned path
  // advances its tap after the last part).
  template <int P = 0, int NP = 1>
  __device__ __forceinline__ void issue(const ConvArgs& a, uint4* lds, int kt, int stage) {
    const int gk = kt_begin + kt;
    uint4* sbase = lds + stage * STAGE_CHUNKS;
    // K tile of the packed weights: gk itself unless taps are skipped
    const int kw_tile = TL ? (ncb * tstride + ntap) * SUBS + nsub : gk;
    if (TL && a.tok) {
      if constexpr (TL) issue_gather<P, NP>(sbase);
    } else if (ALIGNED) {
      const bool kvalid = gk * (8 * KC) < a.K;   // tiles past K (padding to Kp) read zeros
      const int delta = ((nu * a.W + nv) * a.Cs + ncb * 64 + nsub * (8 * KC)) * 2;
#pragma unroll
      for (int j = P; j < RA; j += NP) {
        const int hi = a_hi[j] + nu, wi = a_wi[j] + nv;
        const bool ok = kvalid && (unsigned)hi < (unsigned)a.H && (unsigned)wi < (unsigned)a.W;
        const unsigned off = ok ? (unsigned)(a_off[j] + delta) : oob;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void*)(sbase + (j * NW + wave) * 64), 16, off, 0, 0, 0);
      }
      if (P == NP - 1 && ++nsub == SUBS) {
        nsub = 0;
        if (++ntap == (TL ? taps : a.kh * a.kw)) {
          ntap = 0; nu = 0; nv = 0; ++ncb;
        } else if (++nv == a.kw) {
          nv = 0; ++nu;
        }
      }
    } else {
      const unsigned k8 = (unsigned)(gk * KC + chunk);
      const unsigned tap = a.mag_cs8 ? __umulhi(k8, a.mag_cs8) : k8;
      const int ci = (int)(k8 - tap * a.Cs8) * 8;
      const unsigned u = a.mag_kw ? __umulhi(tap, a.mag_kw) : tap;
      const int v = (int)(tap - u * a.kw);
      const bool kvalid = (int)k8 < a.K8;
#pragma unroll
      for (int j = P; j < RA; j += NP) {
        const int hi = a_hi[j] + (int)u, wi = a_wi[j] + v;
        const bool ok = kvalid && (unsigned)hi < (unsigned)a.H && (unsigned)wi < (unsigned)a.W;
        const unsigned off = ok ? (unsigned)((a_img[j] + hi * a.W + wi) * a.Cs + ci) * 2u : oob;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void*)(sbase + (j * NW + wave) * 64), 16, off, 0, 0, 0);
      }
    }
#pragma unroll
    for (int j = P; j < RB; j += NP)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(wr, (lds_void*)(sbase + BM * KC + (j * NW + wave) * 64), 16,
                                               b_off[j], kw_tile * (KC * 16), 0, 0);
  }
};

// Wait until at most `n` tiles' loads (of `per` instructions each) are outstanding.
template <int PER, int MAXN>
__device__ __forceinline__ void wait_tiles(int n) {
  if constexpr (MAXN >= 1) {
    if (n >= MAXN) {
      wait_vmcnt<MAXN * PER>();
      return;
    }
    wait_tiles<PER, MAXN - 1>(n);
  } else {
    wait_vmcnt<0>();
  }
}

// OCC > 0: registers are limited so that OCC waves fit on each SIMD (more workgroups
// per CU, at the risk of spills).  TAPS: the variant for fused conv1d branches
// (tap_stride > 0, aligned K order only), compiled apart so that the other launches
// keep their own code.
template <int BM, int BN, int WM, int WN, int STAGES, bool ALIGNED, int KC, bool SPLIT, bool SPREAD, int OCC,
          bool TAPS = false>
__global__ __launch_bounds__(WM * WN * 64, OCC > 0 ? OCC : 1) void conv_mfma_kernel(ConvArgs a) {
  use_member(a);
  constexpr int NW = WM * WN;
  constexpr int WTM = BM / WM, WTN = BN / WN;      // wave tile: pixels x channels
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int KS = KC / 2;                       // MFMA k-steps of 16 per K tile
  constexpr bool TL = ALIGNED && TAPS;
  static_assert(!TL || WTM <= 128, "the epilogue max assumes a wave tile spans at most two requests");
  using LoaderT = Loader<BM, BN, NW, ALIGNED, KC, TL>;
  constexpr int PER = LoaderT::RA + LoaderT::RB;   // load instructions per thread per tile
  constexpr int STAGE_CHUNKS = (BM + BN) * KC;     // 16-byte chunks per stage
  static_assert(TM >= 1 && TN >= 1 && LoaderT::RA >= 1 && LoaderT::RB >= 1, "tile shape");
  static_assert(KC == 4 || NW % 2 == 0, "the 64-wide loader's chunk assignment assumes an even wave count");
  static_assert(STAGE_CHUNKS * 16 * STAGES <= 160 * 1024, "LDS budget");
  static_assert(STAGES >= 2 && STAGES <= 6 && (STAGES - 2) * PER < 64, "pipeline depth");
  static_assert(!SPREAD || KS >= 2, "a spread refill needs two k-steps");

  // the ring, or the epilogue's staging of the wave tiles if that is larger
  constexpr int LDS_CHUNKS = STAGES * STAGE_CHUNKS > NW * WTM * 8 ? STAGES * STAGE_CHUNKS : NW * WTM * 8;
  __shared__ uint4 lds[LDS_CHUNKS];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave % WM, wn = wave / WM;
  // Workgroups are dealt round-robin to the 8 XCDs (block b -> XCD b % 8).  Renumber
  // so that each XCD owns a contiguous range of output tiles, walked with the channel
  // tile fastest: the tiles sharing an input tile then run close together on one XCD
  // and read it through that XCD's L2 once.
  const int G = gridDim.x, b = blockIdx.x;
  const int q = G >> 3, r8 = G & 7, xcd = b & 7, loc = b >> 3;
  const int tile = (xcd < r8 ? xcd * (q + 1) : r8 * (q + 1) + (xcd - r8) * q) + loc;
  const int nt = tile % a.n_tiles, mt = tile / a.n_tiles;
  const int m0 = mt * BM, n0 = nt * BN;
  // K tiles that hold any of the K real terms (Kp may pad K by up to 63 with zeros, a
  // whole 32-wide tile of them when KC = 4); skipping a tile of zero products leaves
  // every sum unchanged, bit for bit
  // With fused branches (TL) a tile runs the taps of its widest rows.
  int taps = 0;
  if constexpr (TL) {
    taps = 1;
    const int b0 = n0 / 64, b1 = (n0 + BN - 1) / 64;
#pragma unroll
    for (int b = 0; b < 16; ++b)   // constant indices: the kernel arguments stay in registers
      if (b >= b0 && b <= b1) taps = max(taps, (int)a.taps_by_block[b]);
  }
  const int ktiles = TL ? (a.Cs / 64) * taps * (8 / KC) : (a.K + 8 * KC - 1) / (8 * KC);
  // kt_per_split counts 64-wide tiles, or with fused branches whole channel blocks (of
  // `taps` tiles each), so that a row's products split the same way in every tile
  const int kps = a.kt_per_split * (8 / KC) * (TL ? taps : 1);
  const int kt_begin = blockIdx.y * kps;
  const int nk = min(kps, ktiles - kt_begin);

  LoaderT ld;
  ld.init(a, m0, n0, wave, lane, kt_begin, taps);

  f32x16 acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  const int frow = lane & 31, fk = lane >> 5;
  // Fragment reads: row r of a tile, 16-byte chunk kc (k-step s covers chunks 2s, 2s+1).
  auto frag = [&](const uint4* base, int r, int kc) {
    return __builtin_bit_cast(bf16x8, base[r * KC + (kc ^ swz<KC>(r))]);
  };

  if (nk > 0) {
#pragma unroll
    for (int s = 0; s < STAGES; ++s)
      if (s < nk) ld.issue(a, lds, s, s);
    wait_tiles<PER, STAGES - 1>(min(STAGES, nk) - 1);
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  }

  bf16x8 xf[2][TM], wf[2][TN];
  if (nk > 0) {
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) xf[0][tm] = frag(lds, wm * WTM + tm * 32 + frow, fk);
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) wf[0][tn] = frag(lds + BM * KC, wn * WTN + tn * 32 + frow, fk);
  }

  // Tile t always lives in stage t % STAGES.  The stage freed by tile kt - 1 takes
  // tile kt + STAGES - 1: SPREAD = 0 issues its loads right after the barrier that
  // frees the stage, before the next tile's first fragment reads; SPREAD = 1 issues
  // half of them after the MFMAs of k-step 0 of tile kt and half after those of
  // k-step 1, so that the waves of a large tile do not all stall on a full load
  // queue before their first MFMAs.  Either way they are all issued before the end
  // of tile kt, as the waits assume.
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt % STAGES;
    const uint4* As = lds + cur * STAGE_CHUNKS;
    const uint4* Bs = As + BM * KC;
    const bool refill = SPREAD && kt >= 1 && kt + STAGES - 1 < nk;
    const int rstage = (kt + STAGES - 1) % STAGES;
    const int rt = kt + STAGES - 1;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int b = s & 1;
      if (s < KS - 1) {
        // prefetch the fragments of k-step s + 1 of this tile; the scheduling fence
        // keeps these reads ahead of the MFMAs below, so their latency overlaps them
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) xf[b ^ 1][tm] = frag(As, wm * WTM + tm * 32 + frow, 2 * (s + 1) + fk);
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) wf[b ^ 1][tn] = frag(Bs, wn * WTN + tn * 32 + frow, 2 * (s + 1) + fk);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
          acc[tn][tm] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[b][tn], xf[b][tm], acc[tn][tm], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
      if (refill) {
        if (s == 0) ld.template issue<0, 2>(a, lds, rt, rstage);
        if (s == 1) ld.template issue<1, 2>(a, lds, rt, rstage);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    // All of this tile's fragment reads have completed (their MFMAs consumed them).
    // Wait for tile kt + 1, then let every wave pass: stage `cur` is free for tile
    // kt + STAGES and tile kt + 1 is visible to all.
    if (kt + 1 < nk) {
      asm volatile("" ::: "memory");
      wait_tiles<PER, STAGES - 2>(min(STAGES - 2, nk - 2 - kt));
      __builtin_amdgcn_s_barrier();
      asm volatile("" ::: "memory");
      if (!SPREAD && kt + STAGES < nk) ld.issue(a, lds, kt + STAGES, cur);
      const uint4* An = lds + ((kt + 1) % STAGES) * STAGE_CHUNKS;
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) xf[0][tm] = frag(An, wm * WTM + tm * 32 + frow, fk);
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) wf[0][tn] = frag(An + BM * KC, wn * WTN + tn * 32 + frow, fk);
    }
  }

  // ---- epilogue.  Lane (frow, fk) holds, for each (tn, tm), channels
  // n0 + wn*WTN + tn*32 + 8g + 4fk + j (g, j in 0..3) of pixel m0 + wm*WTM + tm*32 + frow.
  if (SPLIT) {
    // split-K: raw fp32 partial sums, 16-byte stores
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int c = n0 + wn * WTN + tn * 32 + 8 * g + 4 * fk;
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) {
          const int m = m0 + wm * WTM + tm * 32 + frow;
          if (m < a.M)
            *(float4*)(a.partial + ((long long)blockIdx.y * a.M + m) * a.Co_pad + c) =
                make_float4(acc[tn][tm][4 * g + 0], acc[tn][tm][4 * g + 1], acc[tn][tm][4 * g + 2],
                            acc[tn][tm][4 * g + 3]);
        }
      }
    return;
  }
  // Each wave transposes its tile through a private LDS region, 32 channels at a
  // time: the fp32 values acc * scale + shift go to LDS as [pixel][32 channels]
  // (16-byte chunks swizzled by swz(pixel)); each lane then reads 8 channels of one
  // pixel back, adds the residual (16-byte load), applies ReLU, rounds to bf16 and
  // writes 16 bytes.  The residual add and the single rounding match the direct form.
  // A group's residual, scale and shift loads are all issued before its staging
  // writes, so their latency is paid once per group rather than once per pass.
  static_assert(NW * WTM * 32 * 4 <= LDS_CHUNKS * 16, "epilogue staging fits in LDS");
  constexpr int NPASS = WTM / 16;
  const bool bf_res = a.res != nullptr && !a.out_f32;
  float4* stg = (float4*)lds + wave * (WTM * 8);
  const int oq = lane & 3, pl = lane >> 2;   // read phase: channel octet oq of pixel pl (+16 per pass)
  __syncthreads();   // every wave is done with the ring
#pragma unroll
  for (int tn = 0; tn < TN; ++tn) {
    // one 32-channel group at a time: keeps the accumulators in place until used
    __builtin_amdgcn_sched_barrier(0);
    const int cb = n0 + wn * WTN + tn * 32;   // first channel of this 32-channel group
    const int c = cb + 8 * oq;
    uint4 rv[NPASS];
    if (bf_res) {
#pragma unroll
      for (int pass = 0; pass < NPASS; ++pass) {
        const int m = m0 + wm * WTM + pass * 16 + pl;
        rv[pass] = (m < a.M && c < a.c_write) ? *(const uint4*)((const bf16_t*)a.res + (long long)m * a.ldy + c)
                                              : make_uint4(0u, 0u, 0u, 0u);
      }
    }
    float4 sc[4], sh[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      sc[g] = *(const float4*)(a.scale + cb + 8 * g + 4 * fk);
      sh[g] = *(const float4*)(a.shift + cb + 8 * g + 4 * fk);
    }
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int cl = 8 * g + 4 * fk;          // local channel of this lane's 4 values
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) {
        const int p = tm * 32 + frow;
        stg[p * 8 + ((cl >> 2) ^ swz<8>(p))] =
            make_float4(acc[tn][tm][4 * g + 0] * sc[g].x + sh[g].x, acc[tn][tm][4 * g + 1] * sc[g].y + sh[g].y,
                        acc[tn][tm][4 * g + 2] * sc[g].z + sh[g].z, acc[tn][tm][4 * g + 3] * sc[g].w + sh[g].w);
      }
    }
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): this wave's LDS writes have landed
    __builtin_amdgcn_wave_barrier();
    if constexpr (TL) {
      if (a.maxslot) {
        // Max over positions: lane (r, o) = (lane % 16, lane / 16) folds rows
        // pass * 16 + r of channels c .. c + 7 (octet o) into the running max of the
        // wave tile's first request (A) or, if the tile reaches it, the next (B) (a
        // wave tile has at most 128 rows and a request at least 128 positions).  The
        // 16 lanes of one octet form a DPP row and reduce with four DPP steps; lane
        // r = 0 merges the result with atomic max.  The values are the bf16-rounded
        // outputs the stored path would write, so the max is the same.
        const int r = lane & 15, o = lane >> 4;
        const int cm = cb + 8 * o;
        const int mw = m0 + wm * WTM;
        const int nA = mw / a.Wo, rowB = (nA + 1) * a.Wo;
        const bool has_b = rowB < min(mw + WTM, a.M);   // wave-uniform
        int kwb = 1;
#pragma unroll
        for (int b = 0; b < 16; ++b)   // constant indices: the kernel arguments stay in registers
          if (b == (cb >> 6)) kwb = a.taps_by_block[b];
        const int len = a.W - kwb + 1;   // positions of this channel block's branch
        float mA[8], mB[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) mA[j] = mB[j] = -INFINITY;
#pragma unroll
        for (int pass = 0; pass < NPASS; ++pass) {
          const int p = pass * 16 + r;
          const int m = mw + p;
          const float4 lo = stg[p * 8 + ((2 * o) ^ swz<8>(p))];
          const float4 hi = stg[p * 8 + ((2 * o + 1) ^ swz<8>(p))];
          const float v[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
          const bool inB = m >= rowB;
          const int wo = m - (inB ? rowB : rowB - a.Wo);
          if (m >= a.M || wo >= len) continue;
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const float t = bf2f_m(f2bf_m(a.relu ? fmaxf(v[j], 0.f) : v[j]));
            if (inB) mB[j] = fmaxf(mB[j], t);
            else mA[j] = fmaxf(mA[j], t);
          }
        }
        auto row_max = [](float x) {   // max over the 16 lanes of a DPP row, in every lane
          x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, false)));
          x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, false)));
          x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x141, 0xF, 0xF, false)));
          x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x140, 0xF, 0xF, false)));
          return x;
        };
#pragma unroll
        for (int j = 0; j < 8; ++j) mA[j] = row_max(mA[j]);
        if (has_b) {
#pragma unroll
          for (int j = 0; j < 8; ++j) mB[j] = row_max(mB[j]);
        }
        if (r == 0 && cm < a.c_write) {
          unsigned* sA = a.maxslot + (long long)nA * a.ldslot + cm;
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            if (mA[j] > -INFINITY) atomicMax(sA + j, max_key(mA[j]));
            if (has_b && mB[j] > -INFINITY) atomicMax(sA + a.ldslot + j, max_key(mB[j]));
          }
        }
        __builtin_amdgcn_s_waitcnt(0xC07F);   // reads done before the region is rewritten
        __builtin_amdgcn_wave_barrier();
        continue;
      }
    }
    if (a.pool2) {
      // fused 2x2 max-pool: rows 4w .. 4w + 3 of the wave tile form window w; lane
      // (pl, oq) takes window pass * 16 + pl.  The max of the four fp32 values, then
      // ReLU and one rounding, equals the max of the four rounded ReLU outputs.
#pragma unroll
      for (int pass = 0; pass < (WTM / 4 + 15) / 16; ++pass) {
        const int wdw = pass * 16 + pl;
        const int mb = m0 + wm * WTM + 4 * wdw;
        if (4 * wdw >= WTM || mb >= a.M || c >= a.c_write) continue;
        float v[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int p = 4 * wdw + i;
          const float4 lo = stg[p * 8 + ((2 * oq) ^ swz<8>(p))];
          const float4 hi = stg[p * 8 + ((2 * oq + 1) ^ swz<8>(p))];
          const float t[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
#pragma unroll
          for (int j = 0; j < 8; ++j) v[j] = i == 0 ? t[j] : fmaxf(v[j], t[j]);
        }
        if (a.relu) {
#pragma unroll
          for (int j = 0; j < 8; ++j) v[j] = relu_m(v[j]);
        }
        uint4 w;
        w.x = pack2_bf16(v[0], v[1]);
        w.y = pack2_bf16(v[2], v[3]);
        w.z = pack2_bf16(v[4], v[5]);
        w.w = pack2_bf16(v[6], v[7]);
        *(uint4*)((bf16_t*)a.y + (long long)(mb >> 2) * a.ldy + c) = w;
      }
      __builtin_amdgcn_s_waitcnt(0xC07F);   // reads done before the region is rewritten
      __builtin_amdgcn_wave_barrier();
      continue;
    }
#pragma unroll
    for (int pass = 0; pass < NPASS; ++pass) {
      const int p = pass * 16 + pl;
      const int m = m0 + wm * WTM + p;
      const float4 lo = stg[p * 8 + ((2 * oq) ^ swz<8>(p))];
      const float4 hi = stg[p * 8 + ((2 * oq + 1) ^ swz<8>(p))];
      float v[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
      if (m >= a.M || c >= a.c_write) continue;
      const long long o = (long long)m * a.ldy + c;
      if (a.out_f32) {   // fp32 rows (logits): any row stride, element stores
        float* y = (float*)a.y + o;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          if (c + j >= a.c_write) break;
          float t = v[j] + (a.res ? bf2f_m(((const bf16_t*)a.res)[o + j]) : 0.f);
          y[j] = a.relu ? fmaxf(t, 0.f) : t;
        }
        continue;
      }
      if (bf_res) {
        const uint4 r = rv[pass];
        v[0] += bf2f_m(r.x & 0xFFFFu); v[1] += bf2f_m(r.x >> 16);
        v[2] += bf2f_m(r.y & 0xFFFFu); v[3] += bf2f_m(r.y >> 16);
        v[4] += bf2f_m(r.z & 0xFFFFu); v[5] += bf2f_m(r.z >> 16);
        v[6] += bf2f_m(r.w & 0xFFFFu); v[7] += bf2f_m(r.w >> 16);
      }
      if (a.relu) {
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = relu_m(v[j]);
      }
      uint4 w;
      w.x = pack2_bf16(v[0], v[1]);
      w.y = pack2_bf16(v[2], v[3]);
      w.z = pack2_bf16(v[4], v[5]);
      w.w = pack2_bf16(v[6], v[7]);
      *(uint4*)((bf16_t*)a.y + o) = w;
    }
    __builtin_amdgcn_s_waitcnt(0xC07F);   // reads done before the region is rewritten
    __builtin_amdgcn_wave_barrier();
  }
}

template <int BM, int BN, int WM, int WN, int STAGES, int KC, bool SP, int OC>
static hipError_t launch_mfma_cfg(const ConvArgs& a, int splits, hipStream_t s) {
  ConvArgs b = a;
  b.n_tiles = (a.Nc + BN - 1) / BN;
  const int m_tiles = (a.M + BM - 1) / BM;
  if (a.n_members > kMaxGroup) return hipErrorInvalidValue;
  dim3 grid(m_tiles * b.n_tiles, splits, a.n_members > 1 ? a.n_members : 1);
  const dim3 block(WM * WN * 64);
  if (a.tap_stride > 0) {   // fused branches: aligned K order only
    if (a.Cs % 64 != 0) return hipErrorInvalidValue;
    if (splits > 1)
      launch((conv_mfma_kernel<BM, BN, WM, WN, STAGES, true, KC, true, SP, OC, true>), grid, block, s, b);
    else
      launch((conv_mfma_kernel<BM, BN, WM, WN, STAGES, true, KC, false, SP, OC, true>), grid, block, s, b);
  } else if (splits > 1) {
    if (a.Cs % 64 == 0)
      launch((conv_mfma_kernel<BM, BN, WM, WN, STAGES, true, KC, true, SP, OC>), grid, block, s, b);
    else
      launch((conv_mfma_kernel<BM, BN, WM, WN, STAGES, false, KC, true, SP, OC>), grid, block, s, b);
  } else if (a.Cs % 64 == 0) {
    launch((conv_mfma_kernel<BM, BN, WM, WN, STAGES, true, KC, false, SP, OC>), grid, block, s, b);
  } else {
    launch((conv_mfma_kernel<BM, BN, WM, WN, STAGES, false, KC, false, SP, OC>), grid, block, s, b);
  }
  return hipGetLastError();
}

// Sum the split-K partials in split order, then the same epilogue as the GEMM kernel.
// One thread per (output row, 4-channel group); with a fused 2x2 max-pool an output row
// is window q, the max over GEMM rows 4q .. 4q + 3.
__global__ void splitk_reduce_kernel(ConvArgs a, int splits, int in_bf16) {
  use_member(a);
  const int groups = (a.c_write + 3) / 4;
  const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (a.pool2) {
    if (idx >= (long long)(a.M / 4) * groups) return;
    const int q = (int)(idx / groups);
    const int c = (int)(idx - (long long)q * groups) * 4;
    const float4 sc = *(const float4*)(a.scale + c);
    const float4 sh = *(const float4*)(a.shift + c);
    float best[4];
    for (int i = 0; i < 4; ++i) {
      const int m = 4 * q + i;
      float4 s = *(const float4*)(a.partial + (long long)m * a.Co_pad + c);
      for (int z = 1; z < splits; ++z) {
        const float4 t = *(const float4*)(a.partial + ((long long)z * a.M + m) * a.Co_pad + c);
        s.x += t.x; s.y += t.y; s.z += t.z; s.w += t.w;
      }
      const float v[4] = {s.x * sc.x + sh.x, s.y * sc.y + sh.y, s.z * sc.z + sh.z, s.w * sc.w + sh.w};
      for (int j = 0; j < 4; ++j) best[j] = i == 0 ? v[j] : fmaxf(best[j], v[j]);
    }
    const long long o = (long long)q * a.ldy + c;
    for (int j = 0; j < 4; ++j) {
      if (c + j >= a.c_write) break;
      ((bf16_t*)a.y)[o + j] = (bf16_t)f2bf_m(a.relu ? fmaxf(best[j], 0.f) : best[j]);
    }
    return;
  }
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
      if (in_bf16) v[j] += bf2f_m(((const bf16_t*)a.res)[o + j]);
      else v[j] += ((const float*)a.res)[o + j];
    }
  }
  for (int j = 0; j < 4; ++j) {
    if (c + j >= a.c_write) break;
    float t = a.relu ? fmaxf(v[j], 0.f) : v[j];
    if (a.out_f32) ((float*)a.y)[o + j] = t;
    else ((bf16_t*)a.y)[o + j] = (bf16_t)f2bf_m(t);
  }
}

// Tile configurations: id, BM x BN, waves WM x WN, pipeline stages, 16-byte chunks
// per row of a K tile (8: 64 channels, 4: 32 channels; a narrower K tile fits more
// stages in the same LDS), refill schedule (SP = 1: spread over two k-steps).
// Every configuration sums each output's K in the same MFMA order, so the choice
// never changes a result.  Each kernel is instantiated explicitly (the host pass
// does not always emit the launch stub of an implicitly instantiated template).
#define RAFIKI_MFMA_CONFIGS(X)                                                         \
  X(0, 256, 256, 4, 2, 2, 8, 0, 0)  /* 8 waves, wave 64x128, two stages */               \
  X(1, 256, 256, 2, 4, 2, 8, 0, 0)  /* 8 waves, wave 128x64, two stages */               \
  X(2, 256, 128, 2, 4, 3, 8, 0, 0)  /* 8 waves, wave 128x32 */                           \
  X(3, 128, 256, 2, 4, 3, 8, 0, 0)  /* 8 waves, wave 64x64 */                            \
  X(4, 256, 128, 2, 2, 2, 8, 0, 0)  /* wave 128x64, two stages */                        \
  X(5, 128, 128, 2, 2, 3, 8, 0, 0)  /* wave 64x64 */                                     \
  X(6, 64, 128, 1, 4, 3, 8, 0, 0)   /* wave 64x32 */                                     \
  X(7, 128, 64, 2, 2, 3, 8, 0, 0)   /* wave 64x32 */                                     \
  X(8, 64, 64, 2, 2, 3, 8, 0, 0)    /* wave 32x32 */                                     \
  X(9, 32, 128, 1, 4, 3, 8, 0, 0)   /* wave 32x32 */                                     \
  X(10, 128, 32, 4, 1, 3, 8, 0, 0)  /* wave 32x32 */                                     \
  X(11, 256, 64, 4, 1, 3, 8, 0, 0)  /* wave 64x64 */                                     \
  X(12, 64, 64, 2, 2, 2, 8, 0, 0)   /* wave 32x32, two stages (short K) */               \
  X(13, 128, 64, 2, 2, 2, 8, 0, 0)  /* wave 64x32, two stages (short K) */               \
  X(14, 64, 128, 1, 4, 2, 8, 0, 0)  /* wave 64x32, two stages (short K) */               \
  X(15, 128, 128, 2, 2, 2, 8, 0, 0) /* wave 64x64, two stages */                         \
  X(16, 128, 256, 2, 4, 2, 8, 0, 0) /* 8 waves, wave 64x64, two stages */                \
  X(17, 256, 128, 4, 2, 2, 8, 0, 0) /* 8 waves, wave 64x64, two stages */                \
  X(18, 64, 128, 1, 4, 4, 4, 0, 0)  /* 32-wide K tiles: wave 64x32, 4 stages */          \
  X(19, 256, 256, 4, 2, 2, 8, 1, 0) /* as 0, spread refill */                            \
  X(20, 256, 256, 2, 4, 2, 8, 1, 0) /* as 1, spread refill */                            \
  X(21, 256, 128, 2, 4, 3, 8, 1, 0) /* as 2, spread refill */                            \
  X(22, 128, 256, 2, 4, 3, 8, 1, 0) /* as 3, spread refill */                            \
  X(23, 128, 256, 2, 4, 2, 8, 1, 0) /* as 16, spread refill */                           \
  X(24, 256, 128, 4, 2, 2, 8, 1, 0) /* as 17, spread refill */                           \
  X(25, 128, 128, 2, 2, 2, 8, 1, 0) /* as 15, spread refill */                           \
  X(26, 256, 256, 4, 2, 4, 4, 0, 0) /* 8 waves, wave 64x128, 32-wide K, 4 stages */      \
  X(27, 256, 256, 4, 2, 5, 4, 0, 0) /* 8 waves, wave 64x128, 32-wide K, 5 stages */      \
  X(28, 256, 128, 4, 2, 6, 4, 0, 0) /* 8 waves, wave 64x64, 32-wide K, 6 stages */       \
  X(29, 128, 256, 2, 4, 6, 4, 0, 0) /* 8 waves, wave 64x64, 32-wide K, 6 stages */       \
  X(30, 128, 128, 2, 2, 5, 8, 0, 0) /* wave 64x64, 5 stages */                           \
  X(31, 128, 128, 2, 2, 4, 8, 0, 0) /* wave 64x64, 4 stages */                           \
  X(32, 256, 32, 4, 1, 3, 8, 0, 0)  /* wave 64x32 */                                 \
  X(33, 128, 128, 2, 2, 2, 4, 0, 3) /* wave 64x64, 32-wide K, registers for 3 waves per SIMD */ \
  X(34, 128, 128, 2, 2, 3, 4, 0, 3) /* as 33, three stages */                          \
  X(35, 64, 128, 1, 4, 2, 4, 0, 4)  /* wave 64x32, 32-wide K, 4 waves per SIMD */       \
  X(36, 128, 64, 2, 2, 2, 4, 0, 4)  /* wave 64x32, 32-wide K, 4 waves per SIMD */       \
  X(37, 256, 128, 4, 2, 2, 4, 0, 2) /* 8 waves, wave 64x64, 32-wide K */                 \
  X(38, 256, 64, 2, 2, 2, 8, 0, 0)  /* wave 128x32, two stages */                        \
  X(39, 256, 64, 2, 2, 3, 4, 0, 0)  /* wave 128x32, 32-wide K, 3 stages */                \
  X(40, 128, 128, 2, 4, 3, 8, 0, 0) /* 8 waves, wave 64x32, 3 stages */                   \
  X(41, 128, 128, 4, 2, 4, 4, 0, 0) /* 8 waves, wave 32x64, 32-wide K, 4 stages */        \
  X(42, 128, 128, 2, 4, 2, 8, 0, 0) /* 8 waves, wave 64x32, 2 stages */

#define RAFIKI_CFG_ENTRY(id, BM, BN, WM, WN, ST, KC, SP, OC) {BM, BN, WM * WN, ST, KC * 8},
const MfmaConfig kMfmaConfigs[kNumMfmaConfigs] = {RAFIKI_MFMA_CONFIGS(RAFIKI_CFG_ENTRY)};
#undef RAFIKI_CFG_ENTRY

#define RAFIKI_INSTANTIATE(id, BM, BN, WM, WN, ST, KC, SP, OC)                                      \
  template __global__ void conv_mfma_kernel<BM, BN, WM, WN, ST, true, KC, false, SP, OC>(ConvArgs);  \
  template __global__ void conv_mfma_kernel<BM, BN, WM, WN, ST, false, KC, false, SP, OC>(ConvArgs); \
  template __global__ void conv_mfma_kernel<BM, BN, WM, WN, ST, true, KC, true, SP, OC>(ConvArgs);   \
  template __global__ void conv_mfma_kernel<BM, BN, WM, WN, ST, false, KC, true, SP, OC>(ConvArgs);  \
  template __global__ void conv_mfma_kernel<BM, BN, WM, WN, ST, true, KC, false, SP, OC, true>(ConvArgs); \
  template __global__ void conv_mfma_kernel<BM, BN, WM, WN, ST, true, KC, true, SP, OC, true>(ConvArgs);
RAFIKI_MFMA_CONFIGS(RAFIKI_INSTANTIATE)
#undef RAFIKI_INSTANTIATE

hipError_t launch_conv_mfma(const ConvArgs& a, int cfg, int splits, hipStream_t s) {
  switch (cfg) {
#define RAFIKI_CASE(id, BM, BN, WM, WN, ST, KC, SP, OC) \
    case id: return launch_mfma_cfg<BM, BN, WM, WN, ST, KC, SP, OC>(a, splits, s);
    RAFIKI_MFMA_CONFIGS(RAFIKI_CASE)
#undef RAFIKI_CASE
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_splitk_reduce(const ConvArgs& a, int splits, int in_bf16, hipStream_t s) {
  const long long total = (long long)(a.pool2 ? a.M / 4 : a.M) * ((a.c_write + 3) / 4);
  const int threads = 256;
  const long long blocks = (total + threads - 1) / threads;
  if (a.n_members > kMaxGroup) return hipErrorInvalidValue;
  launch(splitk_reduce_kernel, dim3((unsigned)blocks, 1, a.n_members > 1 ? a.n_members : 1), dim3(threads), s, a, splits,
         in_bf16);
  return hipGetLastError();
}

}  // namespace rafiki
