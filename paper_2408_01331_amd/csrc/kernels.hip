// gfx950 (CDNA4) kernels of the fused N-model training step.
//
// LDS-staged MFMA cores with fp32 accumulation serve
//   - the grouped GEMM that runs every Linear layer's forward, data gradient
//     and weight gradient (with the optimizer step fused into its epilogue)
//     for all models of one depth level in one launch: bf16 workgroups of 16
//     waves, each wave a 32x32 tile of v_mfma_f32_32x32x16_bf16 on a 128x128
//     workgroup tile; fp32 workgroups of 4 waves (2x2) of
//     v_mfma_f32_16x16x4_f32 on 64x64;
//   - the implicit-GEMM convolution passes: forward with the bias / ReLU /
//     2x2 max-pool epilogue and data gradient with the un-pool gather, on
//     halo tiles staged in LDS (bf16: 8 waves of v_mfma_f32_32x32x16_bf16
//     blocks, a lane's runs of four accumulator rows holding a pool window;
//     the gathered passes for other shapes: 16x16x32), and the split-K weight
//     gradient (bf16: the GEMM's 32x32x16 core on k-major operands), reduced
//     in split order by a kernel that applies the update.
// A workgroup owns one output tile of one problem (a halo forward workgroup
// may own several consecutive m-tiles); a flat tile table maps blockIdx.x to
// (problem, first tile). Every output element is reduced over k in a
// fixed order that depends only on its own problem's shape, so a model's
// results are bitwise independent of which other models share the launch.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "internal.h"

#ifndef UN_GEMM_DEPTH
#define UN_GEMM_DEPTH 2
#endif
// Waves of one bf16 GEMM workgroup (m x n): 16 waves of 32x32 output each on
// a 128x128 tile. The k loop and the epilogue are latency bound at these
// shapes (M = batch of a few hundred), and 8 waves per SIMD (two workgroups
// per CU) hide that latency best: measured 1.15 ms (4 waves), 1.04 (8), 1.02
// (16) per 64-MLP step.
#ifndef UN_GEMM_WGM
#define UN_GEMM_WGM 4
#endif
#ifndef UN_GEMM_WGN
#define UN_GEMM_WGN 4
#endif
// k-major LDS stages (BK rows of R elements). bf16: no padding; a half-wave
// of transpose reads takes 64 bytes (4 chunks of 16) from each of four
// consecutive rows, and kmaj_bf16 swizzles the 16-byte chunks so that those
// land in four disjoint 64-byte bank windows: rows of >= 128 elements store
// chunk c of row k at c ^ 4*(k % 4); 64-element rows (two rows per 256 bytes
// of banks) at c ^ 4*((k / 2) % 2). With padded rows instead (stride of 8
// banks) the same reads measured twice the LDS cycles (SQ_LDS_BANK_CONFLICT
// half of SQ_LDS_IDX_ACTIVE). fp32: rows padded by 8 elements.
constexpr int KMAJ_PAD_BF16 = 0, KMAJ_PAD_F32 = 8;
template <int LDR>
__device__ __forceinline__ int kmaj_bf16(int k, int col) {
  static_assert(LDR % 128 == 0 || LDR == 64, "rows of 64 or a multiple of 128 elements");
  const int x = LDR == 64 ? ((k >> 1) & 1) << 2 : (k & 3) << 2;
  return k * LDR + (((col >> 3) ^ x) << 3) + (col & 7);
}
#ifndef UN_HALO_WAVES
#define UN_HALO_WAVES 8
#endif
#ifndef UN_LDS_PAD_CHUNKS
#define UN_LDS_PAD_CHUNKS 1
#endif

namespace un {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// ---------------------------------------------------------------------------
// Element helpers
// ---------------------------------------------------------------------------
// fp32 -> bf16, round to nearest, ties to even, a NaN quieted (its top 16
// bits with bit 6 set): gfx950's conversion instruction (v_cvt_pk_bf16_f32),
// which gives the same bits as that integer rounding (add 0x7fff plus the
// kept least significant bit) for every one of the 2^32 inputs (measured).
__device__ __forceinline__ bf16_t f2bf(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }
// two values rounded as f2bf, lo in bits 0-15 and hi in 16-31: one
// instruction for the pair
__device__ __forceinline__ uint32_t f2bf2(float lo, float hi) {
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){lo, hi}, bf16x2));
}
__device__ __forceinline__ float bf2f(bf16_t h) { return __uint_as_float((uint32_t)h << 16); }

template <typename T> struct TT;
template <> struct TT<float> {
  static constexpr int VEC = 4;     // elements per 16 B
  static constexpr int KSTEP = 16;  // k consumed per fragment load
  __device__ static float to_f(float v) { return v; }
  __device__ static float from_f(float v) { return v; }
};
template <> struct TT<bf16_t> {
  static constexpr int VEC = 8;
  static constexpr int KSTEP = 32;
  __device__ static float to_f(bf16_t v) { return bf2f(v); }
  __device__ static bf16_t from_f(float v) { return f2bf(v); }
};

// Element e of a 16-byte vector holding VEC elements of T.
template <typename T> __device__ __forceinline__ float vget(const u32x4& v, int e);
template <> __device__ __forceinline__ float vget<float>(const u32x4& v, int e) {
  return __uint_as_float(v[e]);
}
template <> __device__ __forceinline__ float vget<bf16_t>(const u32x4& v, int e) {
  uint32_t w = v[e >> 1];
  return __uint_as_float((e & 1) ? (w & 0xffff0000u) : (w << 16));
}
// Raw bits of element e (for copying without conversion).
template <typename T> __device__ __forceinline__ uint32_t vbits(const u32x4& v, int e);
template <> __device__ __forceinline__ uint32_t vbits<float>(const u32x4& v, int e) { return v[e]; }
template <> __device__ __forceinline__ uint32_t vbits<bf16_t>(const u32x4& v, int e) {
  uint32_t w = v[e >> 1];
  return (e & 1) ? (w >> 16) : (w & 0xffffu);
}
template <typename T> __device__ __forceinline__ void vset_bits(u32x4& v, int e, uint32_t bits);
template <> __device__ __forceinline__ void vset_bits<float>(u32x4& v, int e, uint32_t bits) { v[e] = bits; }
template <> __device__ __forceinline__ void vset_bits<bf16_t>(u32x4& v, int e, uint32_t bits) {
  uint32_t w = v[e >> 1];
  v[e >> 1] = (e & 1) ? ((w & 0xffffu) | (bits << 16)) : ((w & 0xffff0000u) | (bits & 0xffffu));
}
// Zero elements [valid, VEC).
template <typename T> __device__ __forceinline__ void vmask_tail(u32x4& v, int valid) {
#pragma unroll
  for (int e = 0; e < TT<T>::VEC; ++e)
    if (e >= valid) vset_bits<T>(v, e, 0u);
}
template <typename T> __device__ __forceinline__ T tbits(uint32_t b);
template <> __device__ __forceinline__ float tbits<float>(uint32_t b) { return __uint_as_float(b); }
template <> __device__ __forceinline__ bf16_t tbits<bf16_t>(uint32_t b) { return (bf16_t)b; }
template <typename T> __device__ __forceinline__ uint32_t bits_of(T v);
template <> __device__ __forceinline__ uint32_t bits_of<float>(float v) { return __float_as_uint(v); }
template <> __device__ __forceinline__ uint32_t bits_of<bf16_t>(bf16_t v) { return v; }

__device__ __forceinline__ u32x4 zero4() { return u32x4{0u, 0u, 0u, 0u}; }

// ---------------------------------------------------------------------------
// MFMA core
// ---------------------------------------------------------------------------
// NW waves per workgroup: 4 as 2 x 2 (m x n), 8 as 2 x 4, 16 as 4 x 4.
template <typename T, int BM, int BN, int BK, int NW = 4>
struct Tile {
  static constexpr int VEC = TT<T>::VEC;
  static constexpr int LDK = BK + UN_LDS_PAD_CHUNKS * VEC;  // LDS row stride in elements (16-byte pad chunks)
  static constexpr int WGN = NW == 4 ? 2 : 4, WGM = NW / WGN, NT = 64 * NW;
  static constexpr int WM = BM / WGM, WN = BN / WGN;
  static constexpr int FM = WM / 16, FN = WN / 16;
  static_assert(NW == 4 || NW == 8 || NW == 16, "4, 8 or 16 waves");
  static_assert(FM >= 1 && FN >= 1, "wave tile smaller than one 16x16 block");
  // this wave's first row and column in the tile
  __device__ __forceinline__ static int wave_m() { return ((int)(threadIdx.x >> 6) / WGN) * WM; }
  __device__ __forceinline__ static int wave_n() { return ((int)(threadIdx.x >> 6) % WGN) * WN; }
  static constexpr int A_ELEMS = BM * LDK, B_ELEMS = BN * LDK;
  static_assert(BK % TT<T>::KSTEP == 0, "BK must be a multiple of the MFMA k step");
};

// acc[i][j][r] holds C[wm + 16i + 4*(lane/16) + r][wn + 16j + lane%16].
template <typename T, int BM, int BN, int BK>
__device__ __forceinline__ void mma_block(const T* sA, const T* sB,
                                          f32x4 (&acc)[Tile<T, BM, BN, BK>::FM][Tile<T, BM, BN, BK>::FN]) {
  using TL = Tile<T, BM, BN, BK>;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = (wave >> 1) * TL::WM, wn = (wave & 1) * TL::WN;
  const int lr = lane & 15, lg = lane >> 4;
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int kk = 0; kk < BK; kk += 32) {
      bf16x8 a[TL::FM], b[TL::FN];
#pragma unroll
      for (int i = 0; i < TL::FM; ++i)
        a[i] = __builtin_bit_cast(bf16x8, *(const u32x4*)(sA + (wm + 16 * i + lr) * TL::LDK + kk + 8 * lg));
#pragma unroll
      for (int j = 0; j < TL::FN; ++j)
        b[j] = __builtin_bit_cast(bf16x8, *(const u32x4*)(sB + (wn + 16 * j + lr) * TL::LDK + kk + 8 * lg));
#pragma unroll
      for (int i = 0; i < TL::FM; ++i)
#pragma unroll
        for (int j = 0; j < TL::FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  } else {
    // Lane group g feeds k = kk + 4g + q to the q-th MFMA; over q = 0..3 and
    // the four groups every k of [kk, kk+16) is summed once.
#pragma unroll
    for (int kk = 0; kk < BK; kk += 16) {
      f32x4 a[TL::FM], b[TL::FN];
#pragma unroll
      for (int i = 0; i < TL::FM; ++i) a[i] = *(const f32x4*)(sA + (wm + 16 * i + lr) * TL::LDK + kk + 4 * lg);
#pragma unroll
      for (int j = 0; j < TL::FN; ++j) b[j] = *(const f32x4*)(sB + (wn + 16 * j + lr) * TL::LDK + kk + 4 * lg);
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int i = 0; i < TL::FM; ++i)
#pragma unroll
          for (int j = 0; j < TL::FN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][q], b[j][q], acc[i][j], 0, 0, 0);
    }
  }
}

// k-blocks [kb0, kb1), LDS double-buffered: the global loads of block kb+1
// are in flight while block kb is multiplied out of LDS buffer (kb-kb0)&1,
// then they are written to the other buffer. One barrier per k-block.
// `smem` holds 2 * (A_ELEMS + B_ELEMS) elements of T. (Loaders have two
// register slots; this loop uses slot 0.)
template <typename T, int BM, int BN, int BK, class LA, class LB>
__device__ __forceinline__ void mma_loop(LA& la, LB& lb, int kb0, int kb1, T* smem,
                                         f32x4 (&acc)[Tile<T, BM, BN, BK>::FM][Tile<T, BM, BN, BK>::FN]) {
  using TL = Tile<T, BM, BN, BK>;
  constexpr int STAGE = TL::A_ELEMS + TL::B_ELEMS;
  if (kb0 >= kb1) return;
  la.template load<0>(kb0);
  lb.template load<0>(kb0);
  la.template store<0>(smem);
  lb.template store<0>(smem + TL::A_ELEMS);
  __syncthreads();
  for (int kb = kb0; kb < kb1; ++kb) {
    const int cur = (kb - kb0) & 1;
    const bool more = kb + 1 < kb1;
    if (more) {
      la.template load<0>(kb + 1);
      lb.template load<0>(kb + 1);
    }
    const T* s = smem + cur * STAGE;
    mma_block<T, BM, BN, BK>(s, s + TL::A_ELEMS, acc);
    if (more) {
      T* d = smem + (cur ^ 1) * STAGE;
      la.template store<0>(d);
      lb.template store<0>(d + TL::A_ELEMS);
    }
    __syncthreads();
  }
}

// mma_loop for one loader `ld` that fills a whole stage (both operands).
template <typename T, int BM, int BN, int BK, class L>
__device__ __forceinline__ void mma_loop1(L& ld, int kb0, int kb1, T* smem,
                                          f32x4 (&acc)[Tile<T, BM, BN, BK>::FM][Tile<T, BM, BN, BK>::FN]) {
  using TL = Tile<T, BM, BN, BK>;
  constexpr int STAGE = TL::A_ELEMS + TL::B_ELEMS;
  if (kb0 >= kb1) return;
  ld.template load<0>(kb0);
  ld.template store<0>(smem);
  __syncthreads();
  for (int kb = kb0; kb < kb1; ++kb) {
    const int cur = (kb - kb0) & 1;
    const bool more = kb + 1 < kb1;
    if (more) ld.template load<0>(kb + 1);
    const T* st = smem + cur * STAGE;
    mma_block<T, BM, BN, BK>(st, st + TL::A_ELEMS, acc);
    if (more) ld.template store<0>(smem + (cur ^ 1) * STAGE);
    __syncthreads();
  }
}

// The grouped GEMM's MFMA policy. bf16 runs v_mfma_f32_32x32x16_bf16, which
// sustains about twice the rate of the 16x16x32 form on gfx950 (2.2 vs 1.2
// PFLOP/s with register operands): each of the WGM x WGN waves owns a
// (BM/WGM) x (BN/WGN) tile of 32x32 blocks, acc[I][J][e] holding
//   C[wm + 32I + 8(e/4) + 4(lane/32) + e%4][wn + 32J + lane%32].
// fp32 keeps the 16x16x4 blocks of mma_block. for_groups visits every run of
// four consecutive rows of one column a lane holds: f(row, col, v[4]) in tile
// coordinates. CLD is the row stride (floats) of the epilogue's LDS tile,
// chosen so that a wave's accumulator writes hit 64 distinct banks.
template <typename T, int BM, int BN, int BK, int WGM_ = UN_GEMM_WGM, int WGN_ = UN_GEMM_WGN> struct GemmMma;

// bf16: UN_GEMM_WGM x UN_GEMM_WGN waves (m x n) per workgroup.
template <int BM, int BN, int BK, int WGM_, int WGN_>
struct GemmMma<bf16_t, BM, BN, BK, WGM_, WGN_> {
  static constexpr int WGM = WGM_, WGN = WGN_, NT = 64 * WGM * WGN;
  static constexpr int WM = BM / WGM, WN = BN / WGN, FM = WM / 32, FN = WN / 32;
  static_assert(FM >= 1 && FN >= 1, "wave tile smaller than one 32x32 block");
  static constexpr int LDK = Tile<bf16_t, BM, BN, BK>::LDK;
  static constexpr int LDR_A = BM + KMAJ_PAD_BF16, LDR_B = BN + KMAJ_PAD_BF16;  // k-major row strides
  static constexpr int CLD = BN + 8;
  static_assert(BK % 16 == 0, "BK must be a multiple of 16");
  using Acc = f32x16[FM][FN];
  __device__ __forceinline__ static void zero(Acc& acc) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
  }
  // The 8 k-consecutive operand values of lane (r = lane % 32, k group
  // lane / 32) for tile row `row0 + lane % 32`, k-step kk.
  // Row-major stage [row][LDK]: one 16-byte read.
  __device__ __forceinline__ static bf16x8 frag_row(const bf16_t* s, int row0, int kk) {
    const int lane = threadIdx.x & 63;
    return __builtin_bit_cast(bf16x8, *(const u32x4*)(s + (row0 + (lane & 31)) * LDK + kk + 8 * (lane >> 5)));
  }
  // k-major stage [k][ldr] (chunks swizzled, kmaj_bf16): two LDS transpose
  // reads. In each group of 16 lanes
  // (rows rb..rb+15 of the fragment, k group kg), address lane a points at
  // row k = k0 + a/4, columns rb + 4(a%4) .. +3; lane i then receives
  // stage[k0 + e][rb + i] for e = 0..3 - four consecutive k of its own row.
  template <int LDR>
  __device__ __forceinline__ static bf16x8 frag_kmaj(const bf16_t* s, int row0, int kk) {
    const int lane = threadIdx.x & 63, h = lane >> 4, a = lane & 15;
    const int rb = row0 + 16 * (h & 1) + 4 * (a & 3), k0 = kk + 8 * (h >> 1) + (a >> 2);
    typedef short s4 __attribute__((ext_vector_type(4)));
    const s4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s4*)(s + kmaj_bf16<LDR>(k0, rb)));
    const s4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s4*)(s + kmaj_bf16<LDR>(k0 + 4, rb)));
    const u32x2 l = __builtin_bit_cast(u32x2, lo), u = __builtin_bit_cast(u32x2, hi);
    return __builtin_bit_cast(bf16x8, u32x4{l[0], l[1], u[0], u[1]});
  }
  template <int AM, int BMODE>
  __device__ __forceinline__ static void block(const bf16_t* sA, const bf16_t* sB, Acc& acc) {
    const int wave = threadIdx.x >> 6;
    const int wm = (wave / WGN) * WM, wn = (wave % WGN) * WN;
#pragma unroll
    for (int kk = 0; kk < BK; kk += 16) {
      bf16x8 a[FM], b[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        a[i] = AM == OP_ROW ? frag_row(sA, wm + 32 * i, kk) : frag_kmaj<LDR_A>(sA, wm + 32 * i, kk);
#pragma unroll
      for (int j = 0; j < FN; ++j)
        b[j] = BMODE == OP_ROW ? frag_row(sB, wn + 32 * j, kk) : frag_kmaj<LDR_B>(sB, wn + 32 * j, kk);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  }
  template <class F>
  __device__ __forceinline__ static void for_groups(const Acc& acc, F&& f) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = (wave / WGN) * WM, wn = (wave % WGN) * WN;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          float v[4] = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
          f(wm + 32 * i + 8 * q + 4 * (lane >> 5), wn + 32 * j + (lane & 31), v);
        }
  }
};

template <int BM, int BN, int BK, int WGM_, int WGN_>
struct GemmMma<float, BM, BN, BK, WGM_, WGN_> {
  using TL = Tile<float, BM, BN, BK>;
  static constexpr int NT = 256;
  static constexpr int LDK = TL::LDK;
  static constexpr int LDR_A = BM + KMAJ_PAD_F32, LDR_B = BN + KMAJ_PAD_F32;
  static constexpr int CLD = BN + 4;
  using Acc = f32x4[TL::FM][TL::FN];
  __device__ __forceinline__ static void zero(Acc& acc) {
#pragma unroll
    for (int i = 0; i < TL::FM; ++i)
#pragma unroll
      for (int j = 0; j < TL::FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // Lane (r = lane % 16, g = lane / 16) feeds k = kk + 4g + q to the q-th
  // 16x16x4 MFMA: its four values of tile row row0 + r.
  template <int MODE, int LDR>
  __device__ __forceinline__ static f32x4 frag(const float* s, int row0, int kk) {
    const int lane = threadIdx.x & 63, r = row0 + (lane & 15), k = kk + 4 * (lane >> 4);
    if constexpr (MODE == OP_ROW) return *(const f32x4*)(s + r * LDK + k);
    else return f32x4{s[k * LDR + r], s[(k + 1) * LDR + r], s[(k + 2) * LDR + r], s[(k + 3) * LDR + r]};
  }
  template <int AM, int BMODE>
  __device__ __forceinline__ static void block(const float* sA, const float* sB, Acc& acc) {
    const int wave = threadIdx.x >> 6;
    const int wm = (wave >> 1) * TL::WM, wn = (wave & 1) * TL::WN;
#pragma unroll
    for (int kk = 0; kk < BK; kk += 16) {
      f32x4 a[TL::FM], b[TL::FN];
#pragma unroll
      for (int i = 0; i < TL::FM; ++i) a[i] = frag<AM, LDR_A>(sA, wm + 16 * i, kk);
#pragma unroll
      for (int j = 0; j < TL::FN; ++j) b[j] = frag<BMODE, LDR_B>(sB, wn + 16 * j, kk);
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int i = 0; i < TL::FM; ++i)
#pragma unroll
          for (int j = 0; j < TL::FN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][q], b[j][q], acc[i][j], 0, 0, 0);
    }
  }
  template <class F>
  __device__ __forceinline__ static void for_groups(const Acc& acc, F&& f) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = (wave >> 1) * TL::WM, wn = (wave & 1) * TL::WN;
#pragma unroll
    for (int i = 0; i < TL::FM; ++i)
#pragma unroll
      for (int j = 0; j < TL::FN; ++j) {
        float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
        f(wm + 16 * i + 4 * (lane >> 4), wn + 16 * j + (lane & 15), v);
      }
  }
};

// The GEMM's k loop over nkb k-blocks: LDS double-buffered, and the global
// loads run DEPTH k-blocks ahead in the loaders' DEPTH register slots, so a
// block's load latency is covered by DEPTH blocks of work (with 16 waves a
// slot is one 16-byte vector per operand and thread, so depth is cheap).
// Block kb sits in register slot kb % DEPTH and in LDS buffer kb % 2. Inside
// the loop every load and store is unconditional (loads past the last block
// re-read it and the copies made of them are never read), so the compiler's
// wait counts stay exact. One barrier per k-block.
struct NoTail {
  __device__ __forceinline__ void operator()() const {}
};

template <typename T, int BM, int BN, int BK, int DEPTH, class MM, int AM, int BMODE, class LA, class LB, class Tail>
__device__ __forceinline__ void gemm_loop(LA& la, LB& lb, int nkb, T* smem, typename MM::Acc& acc, Tail&& tail) {
  using TL = Tile<T, BM, BN, BK>;
  constexpr int STAGE = TL::A_ELEMS + TL::B_ELEMS;
  static_assert(DEPTH >= 1 && DEPTH <= 4, "prefetch depth 1 to 4");
  if (nkb <= 0) {
    tail();
    return;
  }
  // slot S takes block b (clamped to the last block)
  auto issue = [&](auto slot, int b) {
    constexpr int S = decltype(slot)::value;
    const int bb = min(b, nkb - 1);
    la.template load<S>(bb);
    lb.template load<S>(bb);
  };
  issue(std::integral_constant<int, 0>{}, 0);
  if constexpr (DEPTH > 1) issue(std::integral_constant<int, 1 % DEPTH>{}, 1);
  if constexpr (DEPTH > 2) issue(std::integral_constant<int, 2 % DEPTH>{}, 2);
  if constexpr (DEPTH > 3) issue(std::integral_constant<int, 3 % DEPTH>{}, 3);
  la.template store<0>(smem);
  lb.template store<0>(smem + TL::A_ELEMS);
  __syncthreads();
  // iteration kb (slot S = kb % DEPTH, LDS buffer kb % 2, both compile-time
  // in the unrolled group below): refill slot S with block kb + DEPTH (for
  // DEPTH 1 with block kb + 1, after the block's own copy has reached LDS),
  // run block kb from LDS, then move block kb + 1 from its slot to LDS.
  auto step = [&](auto pos, int kb) {
    constexpr int U = decltype(pos)::value, S = U % DEPTH, N1 = (U + 1) % DEPTH, BUF = U & 1;
    issue(std::integral_constant<int, S>{}, kb + (DEPTH > 1 ? DEPTH : 1));
    const T* st = smem + BUF * STAGE;
    MM::template block<AM, BMODE>(st, st + TL::A_ELEMS, acc);
    T* d = smem + (BUF ^ 1) * STAGE;
    la.template store<N1>(d);
    lb.template store<N1>(d + TL::A_ELEMS);
    __syncthreads();
  };
  // the last iteration: no block left to load or stage; it starts with the
  // caller's tail() (epilogue loads, whose latency then overlaps the last
  // block while the slot registers are free)
  auto last = [&](auto pos, int kb) {
    constexpr int BUF = decltype(pos)::value & 1;
    tail();
    const T* st = smem + BUF * STAGE;
    MM::template block<AM, BMODE>(st, st + TL::A_ELEMS, acc);
    __syncthreads();
  };
  // a group of G iterations: a multiple of DEPTH (slots) and of 2 (buffers)
  constexpr int G = DEPTH == 1 ? 2 : (DEPTH == 3 ? 6 : DEPTH);
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;
  using I4 = std::integral_constant<int, 4>;
  using I5 = std::integral_constant<int, 5>;
  int kb = 0;
  if constexpr (std::is_same_v<std::decay_t<Tail>, NoTail>) {
    // no tail action: every block in the loop, the last nkb % G after it
    for (; kb + G <= nkb; kb += G) {
      step(I0{}, kb);
      step(I1{}, kb + 1);
      if constexpr (G > 2) {
        step(I2{}, kb + 2);
        step(I3{}, kb + 3);
      }
      if constexpr (G > 4) {
        step(I4{}, kb + 4);
        step(I5{}, kb + 5);
      }
    }
    if (kb < nkb) step(I0{}, kb);
    if (kb + 1 < nkb) step(I1{}, kb + 1);
    if constexpr (G > 2) {
      if (kb + 2 < nkb) step(I2{}, kb + 2);
      if (kb + 3 < nkb) step(I3{}, kb + 3);
    }
    if constexpr (G > 4) {
      if (kb + 4 < nkb) step(I4{}, kb + 4);
    }
    return;
  }
  for (; kb + G < nkb; kb += G) {
    step(I0{}, kb);
    step(I1{}, kb + 1);
    if constexpr (G > 2) {
      step(I2{}, kb + 2);
      step(I3{}, kb + 3);
    }
    if constexpr (G > 4) {
      step(I4{}, kb + 4);
      step(I5{}, kb + 5);
    }
  }
  // the last 1..G blocks (no loop back-edge follows them); the final one
  // without a load or a stage
  if (kb + 1 == nkb) {
    last(I0{}, kb);
    return;
  }
  step(I0{}, kb);
  if (kb + 2 == nkb) {
    last(I1{}, kb + 1);
    return;
  }
  if constexpr (G > 2) {
    step(I1{}, kb + 1);
    if (kb + 3 == nkb) {
      last(I2{}, kb + 2);
      return;
    }
    step(I2{}, kb + 2);
    if (kb + 4 == nkb) {
      last(I3{}, kb + 3);
      return;
    }
  }
  if constexpr (G > 4) {
    step(I3{}, kb + 3);
    if (kb + 5 == nkb) {
      last(I4{}, kb + 4);
      return;
    }
    step(I4{}, kb + 4);
    last(I5{}, kb + 5);
  }
}

template <typename T, int BM, int BN, int BK, int DEPTH, class MM, int AM, int BMODE, class LA, class LB>
__device__ __forceinline__ void gemm_loop(LA& la, LB& lb, int nkb, T* smem, typename MM::Acc& acc) {
  gemm_loop<T, BM, BN, BK, DEPTH, MM, AM, BMODE>(la, lb, nkb, smem, acc, NoTail{});
}

// LDS of one MFMA kernel: the double-buffered operand tiles, reused by the
// epilogue as an fp32 [BM][BN + 8] tile.
template <typename T, int BM, int BN, int BK>
struct Smem {
  using TL = Tile<T, BM, BN, BK>;
  static constexpr int CLD = BN + 8;
  static constexpr size_t MAIN = 2 * (size_t)(TL::A_ELEMS + TL::B_ELEMS) * sizeof(T);
  static constexpr size_t EPI = (size_t)BM * CLD * sizeof(float);
  static constexpr size_t BYTES = MAIN > EPI ? MAIN : EPI;
};

// ---------------------------------------------------------------------------
// Loaders. load(kb) fetches a k-block from global memory into registers,
// store(s) writes it to LDS as [row][k] (k contiguous, row stride LDK).
// ---------------------------------------------------------------------------
// Global memory as seen by the kernels (address space 1: global_load/store
// instead of flat accesses).
template <class T> using gptr = __attribute__((address_space(1))) T*;
template <class T> __device__ __forceinline__ gptr<const T> G(const T* p) { return (gptr<const T>)p; }
template <class T> __device__ __forceinline__ gptr<T> G(T* p) { return (gptr<T>)p; }

// Exact floor(x / d) for 0 <= x < 2^22 and d >= 1 from the correctly rounded
// reciprocal of d, in three full-rate instructions (an integer division takes
// several quarter-rate multiplies): (x + 1/2) / d lies at least 1/(2d) from
// the nearest integer, farther than the rounding of the reciprocal, of 1/(2d)
// and of the fused product can move it for such x.
struct SmallDiv {
  float r, h;
  int d;
  // rv = fl(1/dv), rounded on the host (a correctly rounded division costs
  // a dozen vector instructions); 0.5 fl(1/dv) = fl(0.5/dv) exactly
  __device__ __forceinline__ SmallDiv(int dv, float rv) : r(rv), h(0.5f * rv), d(dv) {}
  __device__ __forceinline__ int q(int x) const { return (int)fmaf((float)x, r, h); }
  // quotient and remainder (x - q d by a 24-bit multiply: q d <= x < 2^22)
  __device__ __forceinline__ int qr(int x, int& rem) const {
    const int qq = q(x);
    rem = x - __mul24(qq, d);
    return qq;
  }
};

// Raw buffer resource over `bytes` bytes from `base`: loads past the end
// return zero (CDNA buffer range checking), so tile rows beyond the matrix need
// no branches. Word 3 is the gfx9-family default (32-bit data format).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  const int n = bytes <= 0 ? 0 : (bytes > 0x7fffffff ? 0x7fffffff : (int)bytes);
  return __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, n, 0x00020000);
}

// Row-major operand with k contiguous: element (row, k) = base[row*ld + k].
// Rows at or beyond rows_valid read as zero through the buffer range check;
// columns at or beyond K are zeroed on the last, partial k-block only.
template <typename T, int ROWS, int BK, int NT = 256, int SLOTS = 2>
struct RowLoader {
  static constexpr int VEC = TT<T>::VEC, VPR = BK / VEC, NV = ROWS * VPR / NT, LDK = BK + UN_LDS_PAD_CHUNKS * VEC;
  static_assert(ROWS * VPR % NT == 0, "tile too small for the workgroup");
  __amdgpu_buffer_rsrc_t rsrc;
  int off[NV];
  int K;
  u32x4 r[SLOTS][NV];
  __device__ __forceinline__ void init(const T* base, int64_t ld, int rows_valid, int K_) {
    K = K_;
    rsrc = make_rsrc(base, (int64_t)rows_valid * ld * (int64_t)sizeof(T));
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      const int v = threadIdx.x + NT * s;
      off[s] = (int)(((int64_t)(v / VPR) * ld + (v % VPR) * VEC) * (int64_t)sizeof(T));
    }
  }
  template <int S>
  __device__ __forceinline__ void load(int kb) {
    const int kbytes = kb * BK * (int)sizeof(T);
#pragma unroll
    for (int s = 0; s < NV; ++s)
      r[S][s] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, off[s] + kbytes, 0, 0));
    if ((kb + 1) * BK > K) {
#pragma unroll
      for (int s = 0; s < NV; ++s) {
        const int k = kb * BK + ((threadIdx.x + NT * s) % VPR) * VEC;
        if (k + VEC > K) vmask_tail<T>(r[S][s], K - k);
      }
    }
  }
  template <int S>
  __device__ __forceinline__ void store(T* sm) const {
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      const int v = threadIdx.x + NT * s;
      *(u32x4*)(sm + (v / VPR) * LDK + (v % VPR) * VEC) = r[S][s];
    }
  }
};

// k-major operand: element (row, k) = mat[k*ld + col0 + row] for the tile
// starting at column col0. A k-block is BK rows of ROWS contiguous elements,
// copied to LDS as they are, [k][ROWS + pad] (bf16: no pad, chunks swizzled
// by kmaj_bf16; the MFMA fragments come out of it through transpose reads).
// The buffer range ends with row K - 1 of the
// matrix, so rows k >= K and anything past the matrix read as zero; columns
// past the tile's valid ones within the matrix only feed output rows /
// columns that are never stored. With bias_col >= 0, column bias_col reads 1
// for every k < K.
template <typename T, int ROWS, int BK, int NT, int SLOTS, int PAD>
struct KRowLoader {
  static constexpr int VEC = TT<T>::VEC, CPR = ROWS / VEC, NV = BK * CPR / NT, LDR = ROWS + PAD;
  static_assert(BK * CPR % NT == 0, "tile too small for the workgroup");
  __amdgpu_buffer_rsrc_t rsrc;
  int off[NV];
  int K, kstride, bias_chunk, bias_e;
  u32x4 r[SLOTS][NV];
  __device__ __forceinline__ void init(const T* mat, int64_t ld, int col0, int K_, int bias_col) {
    K = K_;
    kstride = BK * (int)ld * (int)sizeof(T);
    rsrc = make_rsrc(mat + col0, ((int64_t)K_ * ld - col0) * (int64_t)sizeof(T));
    bias_chunk = bias_col >= 0 ? bias_col / VEC : -1;
    bias_e = bias_col >= 0 ? bias_col % VEC : 0;
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      const int v = threadIdx.x + NT * s;
      off[s] = (int)(((int64_t)(v / CPR) * ld + (v % CPR) * VEC) * (int64_t)sizeof(T));
    }
  }
  template <int S>
  __device__ __forceinline__ void load(int kb) {
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      r[S][s] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, off[s] + kb * kstride, 0, 0));
      const int v = threadIdx.x + NT * s;
      if ((v % CPR) == bias_chunk && kb * BK + v / CPR < K) vset_bits<T>(r[S][s], bias_e, bits_of<T>(TT<T>::from_f(1.0f)));
    }
  }
  template <int S>
  __device__ __forceinline__ void store(T* sm) const {
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      const int v = threadIdx.x + NT * s;
      if constexpr (sizeof(T) == 2) *(u32x4*)(sm + kmaj_bf16<LDR>(v / CPR, (v % CPR) * VEC)) = r[S][s];
      else *(u32x4*)(sm + (v / CPR) * LDR + (v % CPR) * VEC) = r[S][s];
    }
  }
};

// Decode a conv output pixel index into (n, y, x) (pool ordering: m = 4w + d).
__device__ __forceinline__ void decode_out_pixel(const ConvProb& p, int m, int& n, int& y, int& x) {
  if (p.pool) {
    const int w = m >> 2, d = m & 3, pp = p.PH * p.PW;
    n = w / pp;
    const int rem = w - n * pp, ph = rem / p.PW, pw = rem - ph * p.PW;
    y = 2 * ph + (d >> 1);
    x = 2 * pw + (d & 1);
  } else {
    const int pp = p.OH * p.OW;
    n = m / pp;
    const int rem = m - n * pp;
    y = rem / p.OW;
    x = rem - y * p.OW;
  }
}

// Conv forward A operand: rows = output pixels, k = (u, v, c).
template <typename T, int ROWS, int BK>
struct Im2colLoader {
  static constexpr int VEC = TT<T>::VEC, VPR = BK / VEC, NV = ROWS * VPR / 256, LDK = BK + UN_LDS_PAD_CHUNKS * VEC;
  const ConvProb* p;
  const T* X;
  int rn[NV], ry[NV], rx[NV];
  u32x4 r[2][NV];
  __device__ __forceinline__ void init(const ConvProb& pr, int m0) {
    p = &pr;
    X = (const T*)pr.X;
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      const int m = m0 + (threadIdx.x + 256 * s) / VPR;
      int n, y, x;
      decode_out_pixel(pr, m, n, y, x);
      rn[s] = m < pr.M ? n : -1;
      ry[s] = y;
      rx[s] = x;
    }
  }
  template <int S>
  __device__ __forceinline__ void load(int kb) {
    const int C = p->C, H = p->H, W = p->W, KW = p->KH, pad = p->pad, K = p->K;
    const bool vec = (C % VEC) == 0;
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      const int k0 = kb * BK + ((threadIdx.x + 256 * s) % VPR) * VEC;
      u32x4 v = zero4();
      if (rn[s] >= 0 && k0 < K) {
        if (vec) {
          const int t = k0 / C, c = k0 - t * C, u = t / KW, vv = t - u * KW;
          const int y = ry[s] + u - pad, x = rx[s] + vv - pad;
          if (y >= 0 && y < H && x >= 0 && x < W) v = *(const u32x4*)(X + ((int64_t)(rn[s] * H + y) * W + x) * C + c);
        } else {
          // channels not a whole number of vectors: element by element (kept
          // rolled so that the vector paths around it unroll fully)
#pragma unroll 1
          for (int e = 0; e < VEC; ++e) {
            const int k = k0 + e;
            if (k < K) {
              const int t = k / C, c = k - t * C, u = t / KW, vv = t - u * KW;
              const int y = ry[s] + u - pad, x = rx[s] + vv - pad;
              if (y >= 0 && y < H && x >= 0 && x < W)
                vset_bits<T>(v, e, bits_of<T>(X[((int64_t)(rn[s] * H + y) * W + x) * C + c]));
            }
          }
        }
      }
      r[S][s] = v;
    }
  }
  template <int S>
  __device__ __forceinline__ void store(T* sm) const {
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      const int v = threadIdx.x + 256 * s;
      *(u32x4*)(sm + (v / VPR) * LDK + (v % VPR) * VEC) = r[S][s];
    }
  }
};

// dZ[n, p, q, o] of a conv block, gathered from the (already ReLU'-masked)
// gradient at the block output and, with pooling, the window argmax.
// Returns false when (p, q) is outside the conv output or dropped by floor pooling.
__device__ __forceinline__ bool dz_index(const ConvProb& pr, int n, int p, int q, int64_t& idx, int& d) {
  if (p < 0 || q < 0 || p >= pr.OH || q >= pr.OW) return false;
  if (pr.pool) {
    if (p >= 2 * pr.PH || q >= 2 * pr.PW) return false;
    idx = ((int64_t)(n * pr.PH + (p >> 1)) * pr.PW + (q >> 1)) * pr.O;
    d = ((p & 1) << 1) | (q & 1);
  } else {
    idx = ((int64_t)(n * pr.OH + p) * pr.OW + q) * pr.O;
    d = -1;
  }
  return true;
}

// VEC argmax bytes starting at a (VEC-aligned) offset.
template <typename T> __device__ __forceinline__ uint64_t load_am(const uint8_t* a);
template <> __device__ __forceinline__ uint64_t load_am<float>(const uint8_t* a) { return *(gptr<const uint32_t>)a; }
template <> __device__ __forceinline__ uint64_t load_am<bf16_t>(const uint8_t* a) { return *(gptr<const uint64_t>)a; }

// VEC argmax bytes at byte offset off of a buffer resource.
template <typename T> __device__ __forceinline__ uint64_t load_am_buf(__amdgpu_buffer_rsrc_t r, int off);
template <> __device__ __forceinline__ uint64_t load_am_buf<float>(__amdgpu_buffer_rsrc_t r, int off) {
  return (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
}
template <> __device__ __forceinline__ uint64_t load_am_buf<bf16_t>(__amdgpu_buffer_rsrc_t r, int off) {
  const u32x2 v = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0));
  return (uint64_t)v[0] | ((uint64_t)v[1] << 32);
}

// Keep element e of v only where its window argmax equals d.
// The forward pass stores, per window and channel, the byte 1 << (dy*2 + dx)
// of the window's maximum (one-hot), so a selection is a bit test.
template <typename T> __device__ __forceinline__ void select_am(u32x4& v, uint64_t am, int d);
template <> __device__ __forceinline__ void select_am<float>(u32x4& v, uint64_t am, int d) {
#pragma unroll
  for (int e = 0; e < 4; ++e)
    if (!((am >> (8 * e + d)) & 1u)) v[e] = 0u;
}
template <> __device__ __forceinline__ void select_am<bf16_t>(u32x4& v, uint64_t am, int d) {
  // bit d of byte c (element c's byte) is shifted to the top bit of byte c
  // (m1) and of byte c + 1 (m2); the sign-copy selectors of the byte permute
  // (8 / 9: bit 15 / 31 of the second source, 10 / 11: bit 15 / 31 of the
  // first) spread it over the two bytes of element c
  const uint64_t m1 = am << (7 - d), m2 = m1 << 8;
  const uint32_t l1 = (uint32_t)m1, h1 = (uint32_t)(m1 >> 32), l2 = (uint32_t)m2, h2 = (uint32_t)(m2 >> 32);
  v[0] &= __builtin_amdgcn_perm(l1, l2, 0x0A0A0808u);
  v[1] &= __builtin_amdgcn_perm(l1, l2, 0x0B0B0909u);
  v[2] &= __builtin_amdgcn_perm(h1, h2, 0x0A0A0808u);
  v[3] &= __builtin_amdgcn_perm(h1, h2, 0x0B0B0909u);
}
// Is pixel d the maximum of its window (argmax byte a)?
__device__ __forceinline__ bool am_is(uint8_t a, int d) { return (a >> d) & 1u; }

// Conv dgrad A operand: rows = conv input pixels (n, y, x), k = (u, v, o).
template <typename T, int ROWS, int BK>
struct DzGatherLoader {
  static constexpr int VEC = TT<T>::VEC, VPR = BK / VEC, NV = ROWS * VPR / 256, LDK = BK + UN_LDS_PAD_CHUNKS * VEC;
  const ConvProb* p;
  const T* G;
  int rn[NV], ry[NV], rx[NV];
  u32x4 r[2][NV];
  __device__ __forceinline__ void init(const ConvProb& pr, int m0) {
    p = &pr;
    G = (const T*)pr.G;
    const int hw = pr.H * pr.W;
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      // every field written on both sides of the bound (no address select)
      const int m = m0 + (threadIdx.x + 256 * s) / VPR;
      const int n = m / hw, rem = m - n * hw, y = rem / pr.W;
      rn[s] = m < pr.M ? n : -1;
      ry[s] = y;
      rx[s] = rem - y * pr.W;
    }
  }
  template <int S>
  __device__ __forceinline__ void load(int kb) {
    const int O = p->O, KW = p->KH, pad = p->pad, K = p->K;
    const bool vec = (O % VEC) == 0;
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      const int k0 = kb * BK + ((threadIdx.x + 256 * s) % VPR) * VEC;
      u32x4 v = zero4();
      if (rn[s] >= 0 && k0 < K) {
        if (vec) {
          const int t = k0 / O, o = k0 - t * O, u = t / KW, vv = t - u * KW;
          int64_t idx;
          int d;
          if (dz_index(*p, rn[s], ry[s] - u + pad, rx[s] - vv + pad, idx, d)) {
            v = *(const u32x4*)(G + idx + o);
            if (d >= 0) select_am<T>(v, load_am<T>(p->gam + idx + o), d);
          }
        } else {
#pragma unroll 1
          for (int e = 0; e < VEC; ++e) {
            const int k = k0 + e;
            if (k < K) {
              const int t = k / O, o = k - t * O, u = t / KW, vv = t - u * KW;
              int64_t idx;
              int d;
              if (dz_index(*p, rn[s], ry[s] - u + pad, rx[s] - vv + pad, idx, d))
                if (d < 0 || am_is(p->gam[idx + o], d)) vset_bits<T>(v, e, bits_of<T>(G[idx + o]));
            }
          }
        }
      }
      r[S][s] = v;
    }
  }
  template <int S>
  __device__ __forceinline__ void store(T* sm) const {
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      const int v = threadIdx.x + 256 * s;
      *(u32x4*)(sm + (v / VPR) * LDK + (v % VPR) * VEC) = r[S][s];
    }
  }
};

// Conv wgrad operands. Both run along channels in memory while the product
// contracts over pixels, so each thread gathers a VEC-pixel x VEC-channel
// micro-tile (VEC 16-byte vectors, one per pixel), transposes it in registers
// and writes VEC 16-byte LDS rows of VEC consecutive pixels. Threads 0..127
// load A (output channels), threads 128..255 load B (patch columns); a tile
// has exactly 128 micro-tiles per operand for both storage types.

// In-register transpose of a VEC x VEC block: in[p] holds channels 0..VEC-1 of
// pixel p; out[c] receives pixels 0..VEC-1 of channel c.
template <typename T> __device__ __forceinline__ void transpose_block(const u32x4 (&in)[TT<T>::VEC], u32x4 (&out)[TT<T>::VEC]);
template <> __device__ __forceinline__ void transpose_block<float>(const u32x4 (&in)[4], u32x4 (&out)[4]) {
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int p = 0; p < 4; ++p) out[c][p] = in[p][c];
}
template <> __device__ __forceinline__ void transpose_block<bf16_t>(const u32x4 (&in)[8], u32x4 (&out)[8]) {
  // word q of in[p] packs channels (2q, 2q+1) of pixel p (low half = even channel)
#pragma unroll
  for (int q = 0; q < 4; ++q)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const uint32_t a = in[2 * r][q], b = in[2 * r + 1][q];
      out[2 * q][r] = (a & 0xffffu) | (b << 16);
      out[2 * q + 1][r] = (a >> 16) | (b & 0xffff0000u);
    }
}

// Micro-tile of thread t (0..127): 16 row groups x 8 pixel groups. Each run
// of 8 threads takes the 8 pixel groups of one row group, so its 16-byte LDS
// stores (same row, 8 column chunks) fall in distinct banks; the next 8 take
// the adjacent row group (the neighbouring 16 bytes in global memory).
__device__ __forceinline__ void microtile_of(int t, int& rg, int& pg) {
  pg = t & 7;
  rg = ((t >> 3) & 1) | ((t >> 4) << 1);
}

// Weight-gradient operands of one k-block (BK output pixels), both written to
// LDS as [row][pixel]: threads 0..127 build A, rows = output channel o, from
// dZ (the pooled gradient G[w][o], already ReLU'-masked, and the window
// argmax); threads 128..255 build B, rows = j = (u, v, c) plus the bias column
// j == KH*KW*C reading 1, from the input patch in NHWC X. load() only issues
// the global loads into a register slot; the argmax selection, the transpose
// and the LDS writes happen in store(), after the current k-block's products,
// so the loads overlap them. Both roles share the register slots.
// MODE selects the code compiled into the k-loop (a loop body holding every
// path overflows the instruction cache): WG_POOLED / WG_PLAIN for a pooled /
// unpooled block whose channel counts O and C are whole 16-byte vectors,
// WG_GENERIC for anything else (element by element where needed).
enum { WG_GENERIC = 0, WG_POOLED = 1, WG_PLAIN = 2, WG_NARROW = WG_NARROW_BIT };

template <typename T, int BM, int BN, int BK, int MODE>
struct WgradLoader {
  static constexpr int VEC = TT<T>::VEC, NW = VEC / 4, LDK = BK + UN_LDS_PAD_CHUNKS * VEC;
  static constexpr int OOB = 0x7ffffff0;  // a buffer offset past every range: the load returns zero
  static constexpr bool POOL = MODE == WG_POOLED;
  static_assert(BM / VEC == 16 && BN / VEC == 16 && BK / VEC == 8, "16 x 8 micro-tiles per operand");
  static_assert(VEC % 4 == 0, "a micro-tile holds whole 2x2 windows");
  const ConvProb* p;
  bool isA;
  int r0, rg, pg;          // first row (o or j) of this thread's micro-tile
  u32x4 raw[2][VEC];       // A pooled: raw[S][0..NW) = window gradients; else the pixel vectors
  uint64_t am[2][NW];      // A pooled: window argmaxes
  int wkb, wn, wph, wpw;   // B pooled: (image, row, column) of this thread's first window of k-block wkb
  // B generic: column r0 + q's tap offsets (du, dv) and element offset from
  // the pixel's first channel (fixed per thread, so computed once); a column
  // past J gets a dv no pixel brings in range; bq: the bias column's q or -1
  int gdu[VEC], gdv[VEC], goff[VEC], bq;
  __device__ __forceinline__ void init(const ConvProb& pr, int m0, int n0) {
    p = &pr;
    isA = __builtin_amdgcn_readfirstlane(threadIdx.x) < 128;  // waves 0-1: A, waves 2-3: B (wave-uniform)
    microtile_of(threadIdx.x % 128, rg, pg);
    r0 = (isA ? m0 : n0) + rg * VEC;
    wkb = -1;
    if constexpr (MODE == WG_GENERIC) {
      const int C = pr.C, KW = pr.KH, J = pr.KH * pr.KH * C;
      bq = J - r0 >= 0 && J - r0 < VEC ? J - r0 : -1;
#pragma unroll
      for (int q = 0; q < VEC; ++q) {
        const int j = r0 + q;
        if (j < J) {
          const int tq = j / C, c = j - tq * C, uq = tq / KW, vq = tq - uq * KW;
          gdu[q] = uq - pr.pad;
          gdv[q] = vq - pr.pad;
          goff[q] = (gdu[q] * pr.W + gdv[q]) * C + c;
        } else {
          gdu[q] = 0;
          gdv[q] = -(1 << 29);
          goff[q] = 0;
        }
      }
    }
  }
  // advance a pooled window position by `by` windows (row-major over images)
  __device__ __forceinline__ void win_step(int& n, int& ph, int& pw, int by) const {
    pw += by;
    while (pw >= p->PW) {
      pw -= p->PW;
      if (++ph == p->PH) {
        ph = 0;
        ++n;
      }
    }
  }
  __device__ __forceinline__ int64_t out_rows() const {
    return p->pool ? (int64_t)p->Nb * p->PH * p->PW : (int64_t)p->Nb * p->OH * p->OW;
  }
  template <int S>
  __device__ __forceinline__ void load(int kb) {
    if constexpr (MODE == WG_GENERIC) {
      if (isA) loadA_generic<S>(kb);
      else loadB_generic<S>(kb);
    } else {
      if (isA) loadA_fast<S>(kb);
      else loadB_fast<S>(kb);
    }
  }
  // A, whole-vector channels: a micro-tile is entirely below O or entirely past it
  template <int S>
  __device__ __forceinline__ void loadA_fast(int kb) {
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(p->G, out_rows() * p->O * (int64_t)sizeof(T));
    const int O = p->O, o0 = r0, K = p->K;
    const bool rows_in = o0 < O;
    const int pix0 = kb * BK + pg * VEC;
    if constexpr (POOL) {
      const __amdgpu_buffer_rsrc_t rs_am = make_rsrc(p->gam, out_rows() * p->O);
      // VEC consecutive pixels are NW whole windows; past the last pixel or
      // channel: zero gradient and no argmax bit
#pragma unroll
      for (int wq = 0; wq < NW; ++wq) {
        const int pix = pix0 + 4 * wq, idx = (pix >> 2) * O + o0;
        const bool in = rows_in && pix < K;
        raw[S][wq] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, in ? idx * (int)sizeof(T) : OOB, 0, 0));
        am[S][wq] = in ? load_am_buf<T>(rs_am, idx) : 0ull;
      }
    } else {
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const int pix = pix0 + e;
        raw[S][e] = __builtin_bit_cast(
            u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, rows_in && pix < K ? (pix * O + o0) * (int)sizeof(T) : OOB, 0, 0));
      }
    }
  }
  // B, whole-vector channels: a micro-tile's VEC columns are one tap's
  // channels, or the bias chunk (1, 0, ..., 0), or past the bias column
  template <int S>
  __device__ __forceinline__ void loadB_fast(int kb) {
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(p->X, (int64_t)p->Nb * p->H * p->W * p->C * (int64_t)sizeof(T));
    const int C = p->C, H = p->H, W = p->W, KW = p->KH, pad = p->pad, J = p->KH * p->KH * C, j0 = r0;
    const bool bias_chunk = j0 == J, rows_in = j0 < J;
    const int t = j0 / C, c0 = j0 - t * C, u = t / KW, vv = t - u * KW;
    const int pix0 = kb * BK + pg * VEC;
    if constexpr (POOL) {
      // VEC consecutive pixels are NW whole windows; their positions are
      // decoded once and then stepped (k-blocks arrive in order)
      if (kb != wkb) {
        const int w = pix0 >> 2, pp = p->PH * p->PW;
        wn = w / pp;
        const int rem = w - wn * pp;
        wph = rem / p->PW;
        wpw = rem - wph * p->PW;
      }
      int n = wn, ph = wph, pw = wpw;
      win_step(wn, wph, wpw, BK / 4);
      wkb = kb + 1;
#pragma unroll
      for (int wq = 0; wq < NW; ++wq) {
        if (wq > 0) win_step(n, ph, pw, 1);
        const int y0 = 2 * ph, x0 = 2 * pw;
        const bool pin = pix0 + 4 * wq < p->K;
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          const int iy = y0 + (d >> 1) + u - pad, ix = x0 + (d & 1) + vv - pad;
          const bool in = rows_in && pin && iy >= 0 && iy < H && ix >= 0 && ix < W;
          u32x4 val = __builtin_bit_cast(
              u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, in ? (((n * H + iy) * W + ix) * C + c0) * (int)sizeof(T) : OOB, 0, 0));
          if (bias_chunk && pin) vset_bits<T>(val, 0, bits_of<T>(TT<T>::from_f(1.0f)));
          raw[S][4 * wq + d] = val;
        }
      }
    } else {
      // decode the first pixel and step along x
      int n, y, x;
      decode_out_pixel(*p, pix0, n, y, x);
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const bool pin = pix0 + e < p->K;
        const int iy = y + u - pad, ix = x + vv - pad;
        const bool in = rows_in && pin && iy >= 0 && iy < H && ix >= 0 && ix < W;
        u32x4 val = __builtin_bit_cast(
            u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, in ? (((n * H + iy) * W + ix) * C + c0) * (int)sizeof(T) : OOB, 0, 0));
        if (bias_chunk && pin) vset_bits<T>(val, 0, bits_of<T>(TT<T>::from_f(1.0f)));
        raw[S][e] = val;
        if (++x == p->OW) {
          x = 0;
          if (++y == p->OH) {
            y = 0;
            ++n;
          }
        }
      }
    }
  }
  // A, any channel count, pooled or not: final pixel vectors, element by element
  template <int S>
  __device__ __forceinline__ void loadA_generic(int kb) {
    const T* G = (const T*)p->G;
    const int O = p->O, o0 = r0;
    const int pix0 = kb * BK + pg * VEC;
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      const int pix = pix0 + e;
      u32x4 v = zero4();
      if (pix < p->K && o0 < O) {
        const int64_t idx = (int64_t)(p->pool ? (pix >> 2) : pix) * O;
        const int d = p->pool ? (pix & 3) : -1;
#pragma unroll 1
        for (int c = 0; c < VEC; ++c)
          if (o0 + c < O && (d < 0 || am_is(p->gam[idx + o0 + c], d))) vset_bits<T>(v, c, bits_of<T>(G[idx + o0 + c]));
      }
      raw[S][e] = v;
    }
  }
  // B, any channel count, pooled or not: element by element; the pixels'
  // positions decoded once per k-block and stepped (a pooled block's pixels
  // run through each window's four positions, else along the row)
  template <int S>
  __device__ __forceinline__ void loadB_generic(int kb) {
    const gptr<const T> X = G((const T*)p->X);
    const int C = p->C, H = p->H, W = p->W, K = p->K;
    const bool pool = p->pool != 0;
    const int pix0 = kb * BK + pg * VEC;
    int n, y, x;
    decode_out_pixel(*p, pix0, n, y, x);
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      const int pix = pix0 + e;
      u32x4 val = zero4();
      if (pix < K) {
        const int base = ((n * H + y) * W + x) * C;
#pragma unroll
        for (int q = 0; q < VEC; ++q) {
          const int iy = y + gdu[q], ix = x + gdv[q];
          if ((unsigned)iy < (unsigned)H && (unsigned)ix < (unsigned)W)
            vset_bits<T>(val, q, bits_of<T>(X[base + goff[q]]));
        }
#pragma unroll
        for (int q = 0; q < VEC; ++q)
          if (q == bq) vset_bits<T>(val, q, bits_of<T>(TT<T>::from_f(1.0f)));
      }
      raw[S][e] = val;
      if (e + 1 == VEC) break;
      // the next pixel: pooled order (a window's four positions, then the
      // next window), else along the row
      if (pool) {
        if ((pix & 1) == 0) {
          ++x;
        } else if ((pix & 3) == 1) {
          --x;
          ++y;
        } else {
          decode_out_pixel(*p, pix + 1, n, y, x);
        }
      } else if (++x == p->OW) {
        x = 0;
        if (++y == p->OH) {
          y = 0;
          ++n;
        }
      }
    }
  }
  // stage: A tile at stage[0], B tile at stage[BM * LDK]
  template <int S>
  __device__ __forceinline__ void store(T* stage) {
    u32x4 pixv[VEC], out[VEC];
    if (POOL && isA) {
      // each window's gradient lands on its argmax pixel only
#pragma unroll
      for (int wq = 0; wq < NW; ++wq)
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          u32x4 v = raw[S][wq];
          select_am<T>(v, am[S][wq], d);
          pixv[4 * wq + d] = v;
        }
    } else {
#pragma unroll
      for (int e = 0; e < VEC; ++e) pixv[e] = raw[S][e];
    }
    transpose_block<T>(pixv, out);
    T* sm = isA ? stage : stage + BM * LDK;
    const int rl = rg * VEC;
#pragma unroll
    for (int c = 0; c < VEC; ++c) *(u32x4*)(sm + (rl + c) * LDK + pg * VEC) = out[c];
  }
};

// ---------------------------------------------------------------------------
// Grouped NT GEMM
// ---------------------------------------------------------------------------
template <typename T> __device__ __forceinline__ void store_t(void* base, int64_t idx, float v) {
  ((T*)base)[idx] = TT<T>::from_f(v);
}
// element e of a T tensor behind buffer resource r
template <typename T> __device__ __forceinline__ void buf_store_t(__amdgpu_buffer_rsrc_t r, int e, float v);
template <> __device__ __forceinline__ void buf_store_t<float>(__amdgpu_buffer_rsrc_t r, int e, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, e * 4, 0, 0);
}
template <> __device__ __forceinline__ void buf_store_t<bf16_t>(__amdgpu_buffer_rsrc_t r, int e, float v) {
  __builtin_amdgcn_raw_buffer_store_b16(f2bf(v), r, e * 2, 0, 0);
}
// The same at byte offset vb (per lane) + sb (wave-uniform, a scalar operand).
template <typename T> __device__ __forceinline__ void buf_store_ts(__amdgpu_buffer_rsrc_t r, uint32_t vb, int sb, float v);
template <> __device__ __forceinline__ void buf_store_ts<float>(__amdgpu_buffer_rsrc_t r, uint32_t vb, int sb, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, vb, sb, 0);
}
template <> __device__ __forceinline__ void buf_store_ts<bf16_t>(__amdgpu_buffer_rsrc_t r, uint32_t vb, int sb, float v) {
  __builtin_amdgcn_raw_buffer_store_b16(f2bf(v), r, vb, sb, 0);
}

// Load 4 consecutive values (8- or 16-byte aligned) as floats.
template <typename T> __device__ __forceinline__ void load4_t(const T* src, float (&v)[4]);
template <> __device__ __forceinline__ void load4_t<float>(const float* src, float (&v)[4]) {
  const f32x4 x = *(gptr<const f32x4>)src;
  v[0] = x[0];
  v[1] = x[1];
  v[2] = x[2];
  v[3] = x[3];
}
template <> __device__ __forceinline__ void load4_t<bf16_t>(const bf16_t* src, float (&v)[4]) {
  const u32x2 x = *(gptr<const u32x2>)src;
  v[0] = __uint_as_float(x[0] << 16);
  v[1] = __uint_as_float(x[0] & 0xffff0000u);
  v[2] = __uint_as_float(x[1] << 16);
  v[3] = __uint_as_float(x[1] & 0xffff0000u);
}

// Store 4 consecutive values (rows m..m+3 of one column) into a [n][m] array.
template <typename T> __device__ __forceinline__ void store4_t(T* dst, const float (&v)[4], int nvalid) {
  if (nvalid == 4) {
    if constexpr (sizeof(T) == 2) {
      u32x2 w;
      w[0] = f2bf2(v[0], v[1]);
      w[1] = f2bf2(v[2], v[3]);
      *(u32x2*)dst = w;
    } else {
      *(f32x4*)dst = f32x4{v[0], v[1], v[2], v[3]};
    }
  } else {
    for (int r = 0; r < nvalid; ++r) dst[r] = TT<T>::from_f(v[r]);
  }
}

// 16-byte chunk of VE consecutive outputs from fp32 values, as storage type OT.
template <typename OT> __device__ __forceinline__ void store_chunk(OT* dst, const float* v, int nvalid);
template <> __device__ __forceinline__ void store_chunk<float>(float* dst, const float* v, int nvalid) {
  if (nvalid == 4) *(gptr<f32x4>)dst = f32x4{v[0], v[1], v[2], v[3]};
  else
    for (int e = 0; e < nvalid; ++e) G(dst)[e] = v[e];
}
template <> __device__ __forceinline__ void store_chunk<bf16_t>(bf16_t* dst, const float* v, int nvalid) {
  if (nvalid == 8) {
    u32x4 w;
#pragma unroll
    for (int q = 0; q < 4; ++q) w[q] = f2bf2(v[2 * q], v[2 * q + 1]);
    *(gptr<u32x4>)dst = w;
  } else {
    for (int e = 0; e < nvalid; ++e) G(dst)[e] = f2bf(v[e]);
  }
}

// Row-major store of the staged fp32 tile sC [BM][CLD] into C [m][ldc] as OT,
// one 16-byte chunk per thread and step (contiguous along n); the tile rows
// (stride CLD, a multiple of 4) are read as float4s.
// The optimizer step of one element (OptHp): returns the new weight and
// updates the state in place.
__device__ __forceinline__ float opt_update1(const OptHp& h, float g, float w, float* s1, float* s2) {
  if (h.kind == 0.f) return fmaf(-h.lr, g, w);
  if (h.kind == 1.f) {
    const float b = fmaf(h.b1, *s1, g);
    *s1 = b;
    return fmaf(-h.lr, b, w);
  }
  const float m = fmaf(h.b1, *s1, h.c1 * g);
  const float v = fmaf(h.b2, *s2, h.c2 * g * g);
  *s1 = m;
  *s2 = v;
  return w - h.lr * (m / (sqrtf(v) * h.isb2 + h.eps));
}

// Four consecutive elements (16-byte aligned state).
__device__ __forceinline__ void opt_update4(const OptHp& h, const f32x4& g, f32x4& w, float* s1, float* s2) {
  if (h.kind == 0.f) {
#pragma unroll
    for (int e = 0; e < 4; ++e) w[e] = fmaf(-h.lr, g[e], w[e]);
    return;
  }
  f32x4 a = __builtin_nontemporal_load((gptr<const f32x4>)s1);
  if (h.kind == 1.f) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      a[e] = fmaf(h.b1, a[e], g[e]);
      w[e] = fmaf(-h.lr, a[e], w[e]);
    }
    __builtin_nontemporal_store(a, (gptr<f32x4>)s1);
    return;
  }
  f32x4 v = __builtin_nontemporal_load((gptr<const f32x4>)s2);
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    a[e] = fmaf(h.b1, a[e], h.c1 * g[e]);
    v[e] = fmaf(h.b2, v[e], h.c2 * g[e] * g[e]);
    w[e] = w[e] - h.lr * (a[e] / (sqrtf(v[e]) * h.isb2 + h.eps));
  }
  __builtin_nontemporal_store(a, (gptr<f32x4>)s1);
  __builtin_nontemporal_store(v, (gptr<f32x4>)s2);
}

// Column of element (r, c) in the GEMM epilogue's LDS tile: c XOR a multiple
// of 8 that changes every 8 rows. Groups of 8 (float4 pairs) stay contiguous
// for the row passes' float4 reads, and the accumulator writes of a wave
// spread over the banks.
__device__ __forceinline__ int sc_col(int r, int c) { return c ^ (((r >> 3) & 7) << 3); }

// VE consecutive values (one 16-byte vector) as floats.
template <typename T, int VE> __device__ __forceinline__ void load_chunk_f(const T* src, float (&v)[VE]) {
  const u32x4 x = *(gptr<const u32x4>)src;
#pragma unroll
  for (int e = 0; e < VE; ++e) v[e] = vget<T>(x, e);
}

// Row pass of the staged tile: C[m][n] in 16-byte chunks along n. With a
// mask (row-major, same shape), values where the mask is not > 0 become 0
// (ReLU' of the previous layer's output).
template <typename OT, int BM, int BN, int CLD, int NT = 256>
__device__ __forceinline__ void store_rows(const float* sC, OT* C, int64_t ldc, int m0, int n0, int M, int N,
                                           const OT* mask = nullptr, int64_t ldmask = 0,
                                           const OT* add = nullptr, int64_t ldadd = 0, bool relu = false) {
  constexpr int VE = 16 / sizeof(OT), CPR = BN / VE;
  static_assert(CLD % 4 == 0, "float4 rows");
  for (int idx = threadIdx.x; idx < BM * CPR; idx += NT) {
    const int r = idx / CPR, cc = idx - r * CPR;
    const int m = m0 + r, n = n0 + cc * VE;
    if (m >= M || n >= N) continue;
    float v[VE];
#pragma unroll
    for (int e = 0; e < VE; e += 4) {
      const f32x4 x = *(const f32x4*)(sC + r * CLD + sc_col(r, cc * VE + e));
      v[e] = x[0];
      v[e + 1] = x[1];
      v[e + 2] = x[2];
      v[e + 3] = x[3];
    }
    if (add) {
      float av[VE];
      load_chunk_f<OT, VE>(add + (int64_t)m * ldadd + n, av);
#pragma unroll
      for (int e = 0; e < VE; ++e) {
        v[e] += av[e];
        if (relu) v[e] = fmaxf(v[e], 0.f);
      }
    }
    if (mask) {
      float mv[VE];
      load_chunk_f<OT, VE>(mask + (int64_t)m * ldmask + n, mv);
#pragma unroll
      for (int e = 0; e < VE; ++e)
        if (!(mv[e] > 0.f)) v[e] = 0.f;
    }
    store_chunk<OT>(C + (int64_t)m * ldc + n, v, min(VE, N - n));
  }
}

// Softmax cross-entropy of a logits tile staged in LDS (whole rows: N <= BN),
// fused into the logits GEMM: CE_LANES lanes per row reduce max and sum with
// lane shuffles in the same order as ce_rows_kernel, write dL/dz =
// (softmax - onehot) / B to C, and the row losses of the tile are summed in
// row order into ce_part[tm] (a workspace buffer: wsoff bytes added).
template <typename T, int BM, int CLD, int NT>
__device__ __forceinline__ void fused_softmax_ce(float* sC, const GemmProb& p, int m0, int tm,
                                                 const int32_t* __restrict__ labels, int per_model_labels,
                                                 int64_t wsoff) {
  constexpr int RPP = NT / CE_LANES;  // rows per pass
  static_assert(NT % CE_LANES == 0 && BM % RPP == 0, "whole rows per pass");
  __shared__ float s_loss[BM];
  const int sub = threadIdx.x % CE_LANES, C = p.N;
  const float invB = 1.0f / (float)p.M;
  const int32_t* y = labels + (per_model_labels ? p.lab_own : p.lab_shared);
  for (int r0 = 0; r0 < BM; r0 += RPP) {
    const int rl = r0 + (int)threadIdx.x / CE_LANES, b = m0 + rl;
    const bool valid = b < p.M;
    const float* z = sC + rl * CLD;
    float mx = -INFINITY;
    if (valid)
      for (int c = sub; c < C; c += CE_LANES) mx = fmaxf(mx, z[sc_col(rl, c)]);
#pragma unroll
    for (int off = 1; off < CE_LANES; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
    // the exponentials replace the logits in LDS (each lane its own
    // columns), so the gradient pass does not recompute them
    float* ze = sC + rl * CLD;
    float sm = 0.f;
    float zy = 0.f;
    const int yb = valid ? y[b] : 0;
    if (valid) {
      zy = z[sc_col(rl, yb)];
      for (int c = sub; c < C; c += CE_LANES) {
        const float e = expf(z[sc_col(rl, c)] - mx);
        ze[sc_col(rl, c)] = e;
        sm += e;
      }
    }
#pragma unroll
    for (int off = 1; off < CE_LANES; off <<= 1) sm += __shfl_xor(sm, off, 64);
    if (valid) {
      if (sub == 0) s_loss[rl] = mx + logf(sm) - zy;
      const float inv_s = 1.0f / sm;
      T* g = (T*)p.C + (int64_t)b * p.ldc;
      for (int c = sub; c < C; c += CE_LANES)
        g[c] = TT<T>::from_f((ze[sc_col(rl, c)] * inv_s - (c == yb ? 1.f : 0.f)) * invB);
    } else if (sub == 0) {
      s_loss[rl] = 0.f;
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const int nrows = min(BM, p.M - m0);
    float t = 0.f;
    for (int r = 0; r < nrows; ++r) t += s_loss[r];
    ((float*)((char*)p.ce_part + wsoff))[tm] = t;
  }
}

// OPT: the update follows a per-model OptHp (`opt`, not null) instead of
// fma(-lr, g, w); a separate instantiation, so that plain SGD pays nothing.
// BWD: the launch's problems are data gradients (A row-major, B k-major) and
// weight gradients (both k-major), told apart by p.amode; else forward
// problems (both row-major). Each variant compiles only its own k-loops.
template <typename T, int BM, int BN, int BK, bool OPT, bool BWD>
__global__ __launch_bounds__((GemmMma<T, BM, BN, BK>::NT)) __attribute__((amdgpu_waves_per_eu((GemmMma<T, BM, BN, BK>::NT / 128))))
void gemm_kernel(const GemmProb* __restrict__ probs,
                                                   const int32_t* __restrict__ tile_map, float lr,
                                                   const float* __restrict__ lrv, const OptHp* __restrict__ opt,
                                                   int keep_grads, const int32_t* __restrict__ labels,
                                                   int per_model_labels, int64_t wsoff) {
  using TL = Tile<T, BM, BN, BK>;
  using SM = Smem<T, BM, BN, BK>;
  __shared__ __attribute__((aligned(16))) char smem[SM::BYTES];
  const int prob = tile_map[2 * blockIdx.x], local = tile_map[2 * blockIdx.x + 1];
  if (prob < 0) return;  // padding of the XCD-ordered tile list
  const GemmProb& p = probs[prob];
  const int tiles_m = (p.M + BM - 1) / BM;
  int split = 0, tile = local;
  if (p.epi == EPI_WPART) {  // split-K weight gradient: entry = split * tiles + tile
    split = local / (tiles_m * p.tiles_n);
    tile = local - split * (tiles_m * p.tiles_n);
  }
  const int tn = tile / tiles_m, tm = tile - tn * tiles_m;   // m fastest: neighbours share B
  const int m0 = tm * BM, n0 = tn * BN;

  using MM = GemmMma<T, BM, BN, BK>;
  typename MM::Acc acc;
  MM::zero(acc);

  constexpr int NT = MM::NT, D = UN_GEMM_DEPTH;
  constexpr int PAD = sizeof(T) == 2 ? KMAJ_PAD_BF16 : KMAJ_PAD_F32;
  // the k range of this tile: all of K, or the split's chunk (rows kb0 * BK ..)
  const int kb0 = split * p.kchunk;
  const int kc = p.epi == EPI_WPART ? min(p.K - kb0 * BK, p.kchunk * BK) : p.K;
  const int nkb = (kc + BK - 1) / BK;
  constexpr int CPR = BN / 4, NCH = BM * CPR / NT;  // epilogue float4 chunks per row, per thread
  const int ns = p.nsplit;
  f32x4 w0[NCH];  // master weights of the fused update (weight gradient only)
  if constexpr (!BWD) {
    // row-major operands from column k0 on (a split's chunk, else 0), kc of them
    const int64_t k0 = (int64_t)kb0 * BK;
    RowLoader<T, BM, BK, NT, D> la;
    RowLoader<T, BN, BK, NT, D> lb;
    la.init((const T*)p.A + (int64_t)m0 * p.lda + k0, p.lda, p.M - m0, kc);
    lb.init((const T*)p.B + (int64_t)n0 * p.ldb + k0, p.ldb, p.N - n0, kc);
    gemm_loop<T, BM, BN, BK, D, MM, OP_ROW, OP_ROW>(la, lb, nkb, (T*)smem, acc);
  } else if (p.amode == OP_ROW) {
    // data gradient: A = G row-major, B = W k-major (rows k = output units)
    RowLoader<T, BM, BK, NT, D> la;
    KRowLoader<T, BN, BK, NT, D, PAD> lb;
    la.init((const T*)p.A + (int64_t)m0 * p.lda, p.lda, p.M - m0, p.K);
    lb.init((const T*)p.B, p.ldb, n0, p.K, -1);
    gemm_loop<T, BM, BN, BK, D, MM, OP_ROW, OP_KMAJ>(la, lb, nkb, (T*)smem, acc);
  } else {
    // weight gradient: A = G k-major, B = X k-major (rows k = batch), with
    // the ones column of the bias gradient at n == nsplit. The fused
    // update's master-weight loads (this thread's float4 chunks of
    // W[m][n..n+3]) are issued at the start of the k loop's last block, so
    // their latency overlaps that block and the staging below. Master
    // weights, their bf16 copies and the optimizer state are touched once per
    // step: they are loaded and stored non-temporally, so they do not evict
    // the launch's reused operands from L2.
    KRowLoader<T, BM, BK, NT, D, PAD> la;
    KRowLoader<T, BN, BK, NT, D, PAD> lb;
    const int bcol = p.nsplit - n0;
    const int64_t k0 = (int64_t)kb0 * BK;  // k-major: rows k0 .. of both operands
    la.init((const T*)p.A + k0 * p.lda, p.lda, m0, kc, -1);
    lb.init((const T*)p.B + k0 * p.ldb, p.ldb, n0, kc, bcol >= 0 && bcol < BN ? bcol : -1);
    gemm_loop<T, BM, BN, BK, D, MM, OP_KMAJ, OP_KMAJ>(la, lb, nkb, (T*)smem, acc, [&] {
      if (p.epi != EPI_WGRAD) return;
#pragma unroll
      for (int q = 0; q < NCH; ++q) {
        const int idx = threadIdx.x + NT * q, r = idx / CPR, n = n0 + (idx - r * CPR) * 4, m = m0 + r;
        w0[q] = (m < p.M && n + 4 <= ns) ? __builtin_nontemporal_load((gptr<const f32x4>)(p.W + (int64_t)m * p.ldc + n))
                                         : f32x4{0.f, 0.f, 0.f, 0.f};
      }
    });
  }

  // Weight gradient with the update fused: with per-model rates, each tile
  // row's rate goes to LDS.
  __shared__ float s_lr[BM];
  if (p.epi == EPI_WGRAD) {
    if constexpr (!OPT) {
      if (lrv && (int)threadIdx.x < BM) {
        const int m = m0 + threadIdx.x;
        s_lr[threadIdx.x] = m < p.M ? G(lrv)[p.row_model ? G(p.row_model)[m] : p.model] : 0.f;
      }
    }
  }

  // Epilogue 1: per-element work (bias, ReLU) in registers, then the fp32
  // tile to LDS (rows of CLD floats: float4-aligned).
  constexpr int CLD = MM::CLD;
  static_assert(CLD <= SM::CLD, "epilogue tile exceeds its LDS");
  float* sC = (float*)smem;
  const int epi = p.epi;
  MM::for_groups(acc, [&](int rl, int cl, float (&v)[4]) {
      const int mb = m0 + rl, n = n0 + cl;
      const int nv = max(0, min(4, p.M - mb));
      if (n < p.N && nv > 0) {
        if (epi == EPI_FWD || epi == EPI_LOGITS) {
          const float b = p.bias[n];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            v[r] += b;
            if (p.relu && !p.R) v[r] = fmaxf(v[r], 0.f);  // with a skip input: after the sum
          }
        }
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) sC[(rl + r) * CLD + sc_col(rl + r, cl)] = v[r];
  });
  __syncthreads();

  if (epi == EPI_WPART) {
    // this split's partial sums, bias column included, as float4 rows
    float* ws = (float*)((char*)p.ws + wsoff) + (int64_t)split * p.M * p.ldws;
#pragma unroll
    for (int q = 0; q < NCH; ++q) {
      const int idx = threadIdx.x + NT * q, r = idx / CPR, cc = idx - r * CPR;
      const int m = m0 + r, n = n0 + cc * 4;
      if (m >= p.M || n >= p.N) continue;
      const f32x4 g = *(const f32x4*)(sC + r * CLD + sc_col(r, cc * 4));
      float* d = ws + (int64_t)m * p.ldws + n;
      if (n + 4 <= p.N) *(gptr<f32x4>)d = g;
      else
        for (int e = 0; e < p.N - n; ++e) d[e] = g[e];
    }
    return;
  }
  if (epi != EPI_WGRAD) {
    if (!BWD && epi == EPI_LOGITS && p.ce_part) {
      fused_softmax_ce<T, BM, CLD, NT>(sC, p, m0, tm, labels, per_model_labels, wsoff);
      return;
    }
    // Row pass: C[m][n] in 16-byte chunks along n (data gradient: with the
    // previous layer's ReLU' from its stored output), adding the skip input
    // of a residual block first where there is one.
    if (p.C) {
      if (epi == EPI_LOGITS) store_rows<float, BM, BN, CLD, NT>(sC, (float*)p.C, p.ldc, m0, n0, p.M, p.N);
      else if constexpr (!BWD)
        store_rows<T, BM, BN, CLD, NT>(sC, (T*)p.C, p.ldc, m0, n0, p.M, p.N, nullptr, 0, (const T*)p.R, p.ldr,
                                       p.relu && p.R);
      else
        store_rows<T, BM, BN, CLD, NT>(sC, (T*)p.C, p.ldc, m0, n0, p.M, p.N, p.relu ? (const T*)p.mask : nullptr,
                                       p.ldmask, (const T*)p.R, p.ldr);
    }
    return;
  }

  // EPI_WGRAD, SGD fused. Row pass over the float4 chunks: the update, the
  // bf16 copy, the kept gradient. The bias column (n == nsplit) is done
  // element-wise. The master weights this loop reads have all landed before
  // its first store (one wait here): a wait for a load issued before a store
  // still in flight would wait for that store as well, every chunk.
  __builtin_amdgcn_s_waitcnt(0);
#pragma unroll
  for (int q = 0; q < NCH; ++q) {
    const int idx = threadIdx.x + NT * q, r = idx / CPR, cc = idx - r * CPR;
    const int m = m0 + r, n = n0 + cc * 4;
    if (m >= p.M || n > ns) continue;
    // this row's model: its own optimizer, or its own rate (staged in s_lr)
    const int mdl = OPT ? (p.row_model ? p.row_model[m] : p.model) : 0;
    const float lr_m = (!OPT && lrv) ? s_lr[r] : lr;
    float* s = sC + r * CLD + sc_col(r, cc * 4);
    const int64_t base = (int64_t)m * p.ldc + n;
    if (n + 4 <= ns) {
      const f32x4 g = *(const f32x4*)s;
      if (keep_grads) *(gptr<f32x4>)((float*)p.C + base) = g;
      f32x4 w;
      if constexpr (OPT) {
        w = w0[q];
        opt_update4(opt[mdl], g, w, p.s1 + base, p.s2 + base);
      } else {
        w = f32x4{fmaf(-lr_m, g[0], w0[q][0]), fmaf(-lr_m, g[1], w0[q][1]), fmaf(-lr_m, g[2], w0[q][2]),
                  fmaf(-lr_m, g[3], w0[q][3])};
      }
      __builtin_nontemporal_store(w, (gptr<f32x4>)(p.W + base));
      if (p.Wb) {
        u32x2 hb;
        hb[0] = f2bf2(w[0], w[1]);
        hb[1] = f2bf2(w[2], w[3]);
        __builtin_nontemporal_store(hb, (gptr<u32x2>)((bf16_t*)p.Wb + base));
      }
    } else {
      for (int e = 0; e < 4 && n + e <= ns && n + e < p.N; ++e) {
        const float g = s[e];
        if (n + e < ns) {
          if (keep_grads) ((float*)p.C)[base + e] = g;
          float w;
          if constexpr (OPT) w = opt_update1(opt[mdl], g, p.W[base + e], p.s1 + base + e, p.s2 + base + e);
          else w = fmaf(-lr_m, g, p.W[base + e]);
          p.W[base + e] = w;
          if (p.Wb) ((bf16_t*)p.Wb)[base + e] = f2bf(w);
        } else {
          if (keep_grads) p.dbias[m] = g;
          if constexpr (OPT) p.bmaster[m] = opt_update1(opt[mdl], g, p.bmaster[m], p.sb1 + m, p.sb2 + m);
          else p.bmaster[m] = fmaf(-lr_m, g, p.bmaster[m]);
        }
      }
    }
  }
}

// Zero the elements of v whose element of x is not > 0 (ReLU', x the stored
// output). bf16: two elements per 32-bit word with packed 16-bit integer
// operations: x > 0 exactly when its bits lie in [0x0001, 0x7f80] (positive,
// not NaN), i.e. when 0x7f80 - (x - 1), saturating at 0, is not 0.
template <typename T> __device__ __forceinline__ void relu_mask(u32x4& v, const u32x4& x);
template <> __device__ __forceinline__ void relu_mask<float>(u32x4& v, const u32x4& x) {
#pragma unroll
  for (int e = 0; e < 4; ++e)
    if (!(__uint_as_float(x[e]) > 0.f)) v[e] = 0u;
}
// (each word passed by value: bit-casting the vector's elements in place
// produced one mask for all four words)
__device__ __forceinline__ uint32_t relu_mask_word(uint32_t xw) {
  typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
  const u16x2 one = {1, 1}, top = {0x7f80, 0x7f80}, zero = {0, 0};
  const u16x2 xv = __builtin_bit_cast(u16x2, xw);
  const u16x2 pos = __builtin_elementwise_min(__builtin_elementwise_sub_sat(top, xv - one), one);  // 1 where x > 0
  return __builtin_bit_cast(uint32_t, zero - pos);
}
template <> __device__ __forceinline__ void relu_mask<bf16_t>(u32x4& v, const u32x4& x) {
  const uint32_t x0 = x[0], x1 = x[1], x2 = x[2], x3 = x[3];
  v[0] &= relu_mask_word(x0);
  v[1] &= relu_mask_word(x1);
  v[2] &= relu_mask_word(x2);
  v[3] &= relu_mask_word(x3);
}

// ---------------------------------------------------------------------------
// Convolution passes
// ---------------------------------------------------------------------------
// The conv data-gradient epilogue stages the tile in LDS (after the main
// loop's last barrier) and writes whole 16-byte vectors along the channels.
template <typename T, int BM, int BN>
struct ConvEpiSmem {
  static constexpr int VE = 16 / (int)sizeof(T);          // elements per 16-byte vector
  static constexpr int SLD = BN + VE;                      // staged row stride (elements)
  static constexpr size_t BYTES = (size_t)BM * SLD * sizeof(T);
};

// Accumulator layouts of the conv passes. for_groups(acc, f) visits every run
// of four consecutive tile rows of one column that a lane holds:
// f(row, col, j, v[4]) in tile coordinates, j the lane's column fragment
// (col == col_of(j)).
// Acc16: the 16x16 MFMA blocks of Tile (acc[i][j][r] holds
// C[wm + 16i + 4*(lane/16) + r][wn + 16j + lane%16]).
template <typename T, int BM, int BN, int BK, int NW>
struct Acc16 {
  using TL = Tile<T, BM, BN, BK, NW>;
  static constexpr int FM = TL::FM, FN = TL::FN, NT = TL::NT, ROWS = BM;
  using Acc = f32x4[FM][FN];
  __device__ __forceinline__ static void zero(Acc& acc) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  __device__ __forceinline__ static int col_of(int j) { return TL::wave_n() + 16 * j + (threadIdx.x & 15); }
  // the tile row whose A operand this lane supplies to fragment row i
  __device__ __forceinline__ static int arow(int i) { return TL::wave_m() + 16 * i + (threadIdx.x & 15); }
  template <class F>
  __device__ __forceinline__ static void for_groups(const Acc& acc, F&& f) {
    const int lane = threadIdx.x & 63, wm = TL::wave_m();
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
        f(wm + 16 * i + 4 * (lane >> 4), col_of(j), j, v);
      }
  }
  // the same groups, first row lrow + urow: lrow per lane, urow a constant
  // of the unrolled loop
  template <class F>
  __device__ __forceinline__ static void for_groups_split(const Acc& acc, F&& f) {
    const int lane = threadIdx.x & 63, lrow = TL::wave_m() + 4 * (lane >> 4);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
        f(lrow, 16 * i, col_of(j), j, v);
      }
  }
};

// Acc32 (bf16 halo tiles): 32x32x16 MFMA blocks, each wave 32 columns wide
// (BN / 32 waves across, the rest down): acc[i][e] holds
// C[wm + 32i + 8(e/4) + 4(lane/32) + e%4][wn + lane%32]. A lane's runs of
// four rows start at multiples of four, so a pooled tile's windows stay whole.
template <int BM, int BN, int NW>
struct Acc32 {
  static constexpr int WGN = BN / 32, WGM = NW / WGN, WM = BM / WGM, FM = WM / 32, FN = 1, NT = 64 * NW, ROWS = BM;
  static_assert(WGN >= 1 && WGM >= 1 && WGM * WGN == NW && FM >= 1 && FM * 32 * WGM == BM, "32x32 wave tiles");
  using Acc = f32x16[FM];
  __device__ __forceinline__ static int wave_m() { return ((int)(threadIdx.x >> 6) / WGN) * WM; }
  __device__ __forceinline__ static int wave_n() { return ((int)(threadIdx.x >> 6) % WGN) * 32; }
  __device__ __forceinline__ static void zero(Acc& acc) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][e] = 0.f;
  }
  __device__ __forceinline__ static int col_of(int) { return wave_n() + (threadIdx.x & 31); }
  __device__ __forceinline__ static int arow(int i) { return wave_m() + 32 * i + (threadIdx.x & 31); }
  template <class F>
  __device__ __forceinline__ static void for_groups(const Acc& acc, F&& f) {
    const int lane = threadIdx.x & 63, wm = wave_m();
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float v[4] = {acc[i][4 * q], acc[i][4 * q + 1], acc[i][4 * q + 2], acc[i][4 * q + 3]};
        f(wm + 32 * i + 8 * q + 4 * (lane >> 5), col_of(0), 0, v);
      }
  }
  // the same groups, first row lrow + urow: lrow per lane, urow a constant
  // of the unrolled loop
  template <class F>
  __device__ __forceinline__ static void for_groups_split(const Acc& acc, F&& f) {
    const int lane = threadIdx.x & 63, lrow = wave_m() + 4 * (lane >> 5);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float v[4] = {acc[i][4 * q], acc[i][4 * q + 1], acc[i][4 * q + 2], acc[i][4 * q + 3]};
        f(lrow, 32 * i + 8 * q, col_of(0), 0, v);
      }
  }
};

// Conv forward epilogue: ReLU, 2x2 max-pool in registers (pool rows are
// window-ordered, so a lane's four accumulator rows are one window), then the
// pooled value and its one-hot argmax, stored straight from registers
// (staging this small output in LDS measured slower). One straight-line
// variant per (ReLU, pool, skip input) pattern, chosen by a uniform branch.
//
// Pooling takes the maximum of the raw sums, then adds the bias and applies
// the ReLU once: rounding a + b is monotone in a, so the pooled value is
// fl(max a + b) either way, and the ReLU commutes with the maximum. The
// argmax is the first maximum in (dy, dx) order of the raw sums (two sums
// that differ but round to the same value with the bias pick the larger),
// and the first member (byte 1) where the pooled value is <= 0: the ReLU'd
// window is then all zeros.
// pool4 returns the window's maximum plus the bias, before the ReLU
// (store_relu applies it), and its argmax byte.
template <bool RELU>
__device__ __forceinline__ float pool4(const float (&v)[4], float b, uint32_t& am) {
  am = 1u;
  float mx = v[0];
#pragma unroll
  for (int r = 1; r < 4; ++r)
    if (v[r] > mx) {
      mx = v[r];
      am = 1u << r;
    }
  mx += b;
  if constexpr (RELU) am = mx > 0.f ? am : 1u;
  return mx;
}

// ReLU of two packed bf16 values, on their bits: a negative value (sign bit
// set) is a negative 16-bit integer. Rounding commutes with it: rounding is
// monotone and keeps the sign.
__device__ __forceinline__ uint32_t relu_bf16x2(uint32_t w) {
  typedef short s16x2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(s16x2, w), (s16x2){0, 0}));
}

// Store v, after the ReLU if RELU, at byte offset vb + sb.
template <typename T, bool RELU>
__device__ __forceinline__ void store_relu(__amdgpu_buffer_rsrc_t r, uint32_t vb, int sb, float v) {
  if constexpr (sizeof(T) == 2) {
    uint32_t w = f2bf2(v, 0.f);
    if constexpr (RELU) w = relu_bf16x2(w);
    __builtin_amdgcn_raw_buffer_store_b16((uint16_t)w, r, vb, sb, 0);
  } else {
    buf_store_ts<T>(r, vb, sb, RELU ? fmaxf(v, 0.f) : v);
  }
}

template <typename T, class L, bool RELU, bool POOL, bool RES>
__device__ __forceinline__ void conv_fwd_epi(const ConvProb& p, int m0, int n0, const typename L::Acc& acc) {
  // the problem's fields as values: read through the problem reference,
  // every field would be loaded again after each store (the stores might
  // alias it)
  const int O = p.O, M = p.M;
  // outputs through buffer stores: 32-bit offsets (tensors are under 2^31
  // bytes), no 64-bit address arithmetic per store
  const __amdgpu_buffer_rsrc_t rP = make_rsrc(p.P, 0x7fffffff), rAM = make_rsrc(p.amax, 0x7fffffff);
  // this lane's biases, loaded before the first store: loads and stores
  // share one in-order counter, so a load issued after the stores would wait
  // for all of them (once per fragment row)
  const gptr<const float> BIAS = G(p.bias);
  float bias[L::FN];
#pragma unroll
  for (int j = 0; j < L::FN; ++j) {
    const int o = n0 + L::col_of(j);
    bias[j] = o < O ? BIAS[o] : 0.f;
  }
  if (!RES && m0 + L::ROWS <= M) {
    // a whole tile: no row test. A lane's stores sit at a fixed offset of
    // its own plus a uniform one per group (the scalar operand); lanes past
    // column O store past the buffer's range, where the store is dropped.
    constexpr uint32_t OUT = 0x80000000u;
    L::for_groups_split(acc, [&](int lrow, int urow, int cl, int j, const float (&a)[4]) {
      const int o = n0 + cl;
      float v[4] = {a[0], a[1], a[2], a[3]};
      if constexpr (POOL) {
        // window (m0 + lrow + urow) / 4; 24-bit multiplies (pixel and
        // channel counts are under 2^24)
        const uint32_t e = (uint32_t)(__mul24((m0 + lrow) >> 2, O) + o);
        const int se = (urow >> 2) * O;
        uint32_t am;
        const float mx = pool4<RELU>(v, bias[j], am);
        store_relu<T, RELU>(rP, o < O ? e * (uint32_t)sizeof(T) : OUT, se * (int)sizeof(T), mx);
        __builtin_amdgcn_raw_buffer_store_b8((uint8_t)am, rAM, o < O ? e : OUT, se, 0);
      } else {
        const uint32_t e = (uint32_t)(__mul24(m0 + lrow, O) + o), vb = o < O ? e * (uint32_t)sizeof(T) : OUT;
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] += bias[j];
        if constexpr (sizeof(T) == 2) {
          // two rows per conversion; the second from the high half
#pragma unroll
          for (int r = 0; r < 4; r += 2) {
            uint32_t w = f2bf2(v[r], v[r + 1]);
            if constexpr (RELU) w = relu_bf16x2(w);
            __builtin_amdgcn_raw_buffer_store_b16((uint16_t)w, rP, vb, (urow + r) * O * 2, 0);
            __builtin_amdgcn_raw_buffer_store_b16((uint16_t)(w >> 16), rP, vb, (urow + r + 1) * O * 2, 0);
          }
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            if constexpr (RELU) v[r] = fmaxf(v[r], 0.f);
            buf_store_ts<T>(rP, vb, (urow + r) * O * (int)sizeof(T), v[r]);
          }
        }
      }
    });
    return;
  }
  const gptr<const T> R = G((const T*)p.R);
  L::for_groups(acc, [&](int rl, int cl, int j, const float (&a)[4]) {
    const int mb = m0 + rl, o = n0 + cl;
    if (mb >= M || o >= O) return;
    float v[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      v[r] = POOL ? a[r] : a[r] + bias[j];
      // skip input of a residual block (never pooled): rows are pixels
      if constexpr (RES) v[r] += mb + r < M ? TT<T>::to_f(R[__mul24(mb + r, O) + o]) : 0.f;
      if constexpr (RELU && !POOL) v[r] = fmaxf(v[r], 0.f);
    }
    if constexpr (POOL) {
      // rows mb..mb+3 are one 2x2 window
      uint32_t am;
      const float mx = pool4<RELU>(v, bias[j], am);
      const int e = __mul24(mb >> 2, O) + o;
      store_relu<T, RELU>(rP, (uint32_t)e * (uint32_t)sizeof(T), 0, mx);
      __builtin_amdgcn_raw_buffer_store_b8((uint8_t)am, rAM, e, 0, 0);
    } else {
      const int nv = min(4, M - mb);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        if (r >= nv) break;
        buf_store_t<T>(rP, __mul24(mb + r, O) + o, v[r]);
      }
    }
  });
}

template <typename T, class L>
__device__ __forceinline__ void conv_fwd_epilogue(const ConvProb& p, int m0, int n0, const typename L::Acc& acc) {
  const bool relu = p.relu != 0;
  if (p.R) {  // residual blocks are never pooled
    if (relu) conv_fwd_epi<T, L, true, false, true>(p, m0, n0, acc);
    else conv_fwd_epi<T, L, false, false, true>(p, m0, n0, acc);
  } else if (p.pool) {
    if (relu) conv_fwd_epi<T, L, true, true, false>(p, m0, n0, acc);
    else conv_fwd_epi<T, L, false, true, false>(p, m0, n0, acc);
  } else {
    if (relu) conv_fwd_epi<T, L, true, false, false>(p, m0, n0, acc);
    else conv_fwd_epi<T, L, false, false, false>(p, m0, n0, acc);
  }
}

// Conv data-gradient epilogue: the previous block's ReLU' (its stored output
// > 0) and the store of the gradient at that output, in 16-byte vectors.
template <typename T, int BM, int BN, class L>
__device__ __forceinline__ void conv_dgrad_epilogue(const ConvProb& p, int m0, int n0, const typename L::Acc& acc,
                                                    char* smem) {
  using ES = ConvEpiSmem<T, BM, BN>;
  constexpr int VE = ES::VE, CPR = BN / VE, NT = L::NT;
  const int C = p.C, M = p.M;
  const bool prev_relu = p.prev_relu != 0;
  const gptr<const T> R = G((const T*)p.R);
  const gptr<const T> X = G((const T*)p.X);
  const gptr<T> Gp = G((T*)p.Gprev);
  T* sG = (T*)smem;
  L::for_groups(acc, [&](int rl, int cl, int, const float (&a)[4]) {
    if (R) {
      // gradient at a residual block's output joins before the rounding
      const int c = n0 + cl;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + rl + r;
        const float add = (m < M && c < C) ? TT<T>::to_f(R[m * C + c]) : 0.f;
        sG[(rl + r) * ES::SLD + cl] = TT<T>::from_f(a[r] + add);
      }
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r) sG[(rl + r) * ES::SLD + cl] = TT<T>::from_f(a[r]);
    }
  });
  __syncthreads();
  const bool vec = (C % VE) == 0;
  if (vec) {
    // the ReLU' chunks of all of this thread's steps before its first store
    // (loads and stores share one in-order counter)
    constexpr int NI = (BM * CPR + NT - 1) / NT;
    u32x4 xs[NI];
#pragma unroll
    for (int s = 0; s < NI; ++s) {
      const int idx = threadIdx.x + NT * s, r = idx / CPR, c = n0 + (idx - r * CPR) * VE, m = m0 + r;
      xs[s] = (prev_relu && idx < BM * CPR && m < M && c < C) ? *(gptr<const u32x4>)(X + m * C + c) : zero4();
    }
#pragma unroll
    for (int s = 0; s < NI; ++s) {
      const int idx = threadIdx.x + NT * s, r = idx / CPR, c = n0 + (idx - r * CPR) * VE, m = m0 + r;
      if (idx >= BM * CPR || m >= M || c >= C) continue;
      u32x4 v = *(const u32x4*)(sG + r * ES::SLD + (c - n0));
      if (prev_relu) relu_mask<T>(v, xs[s]);
      *(gptr<u32x4>)(Gp + m * C + c) = v;
    }
    return;
  }
  for (int idx = threadIdx.x; idx < BM * CPR; idx += NT) {
    const int r = idx / CPR, c = n0 + (idx - r * CPR) * VE, m = m0 + r;
    if (m >= M || c >= C) continue;
    const int g = m * C + c;
    const T* sv = sG + r * ES::SLD + (c - n0);
    for (int e = 0; e < VE && c + e < C; ++e) {
      T v = sv[e];
      if (prev_relu && !(TT<T>::to_f(X[g + e]) > 0.f)) v = TT<T>::from_f(0.f);
      Gp[g + e] = v;
    }
  }
}

template <typename T, int BM, int BN, int BK>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void conv_fwd_kernel(const ConvProb* __restrict__ probs,
                                                       const int32_t* __restrict__ tile_map) {
  using TL = Tile<T, BM, BN, BK>;
  __shared__ __attribute__((aligned(16))) char smem[Smem<T, BM, BN, BK>::BYTES];
  const int prob = tile_map[2 * blockIdx.x], local = tile_map[2 * blockIdx.x + 1];
  if (prob < 0) return;  // padding of the XCD-ordered tile list
  const ConvProb& p = probs[prob];
  const int tm = local / p.tiles_n, tn = local - tm * p.tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;

  using L = Acc16<T, BM, BN, BK, 4>;
  typename L::Acc acc;
  L::zero(acc);

  Im2colLoader<T, BM, BK> la;
  la.init(p, m0);
  RowLoader<T, BN, BK> lb;
  lb.init((const T*)p.Wt + (int64_t)n0 * p.ldw, p.ldw, p.N - n0, p.K);
  mma_loop<T, BM, BN, BK>(la, lb, 0, (p.K + BK - 1) / BK, (T*)smem, acc);

  conv_fwd_epilogue<T, L>(p, m0, n0, acc);
}

template <typename T, int BM, int BN, int BK>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void conv_dgrad_kernel(const ConvProb* __restrict__ probs,
                                                         const int32_t* __restrict__ tile_map) {
  using TL = Tile<T, BM, BN, BK>;
  __shared__ __attribute__((aligned(16))) char smem[Smem<T, BM, BN, BK>::BYTES];
  const int prob = tile_map[2 * blockIdx.x], local = tile_map[2 * blockIdx.x + 1];
  if (prob < 0) return;  // padding of the XCD-ordered tile list
  const ConvProb& p = probs[prob];
  const int tm = local / p.tiles_n, tn = local - tm * p.tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;

  f32x4 acc[TL::FM][TL::FN];
#pragma unroll
  for (int i = 0; i < TL::FM; ++i)
#pragma unroll
    for (int j = 0; j < TL::FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  DzGatherLoader<T, BM, BK> la;
  la.init(p, m0);
  RowLoader<T, BN, BK> lb;
  lb.init((const T*)p.Wt + (int64_t)n0 * p.ldw, p.ldw, p.N - n0, p.K);
  mma_loop<T, BM, BN, BK>(la, lb, 0, (p.K + BK - 1) / BK, (T*)smem, acc);

  conv_dgrad_epilogue<T, BM, BN, Acc16<T, BM, BN, BK, 4>>(p, m0, n0, acc, smem);
}

// ---------------------------------------------------------------------------
// Halo-tiled implicit-GEMM convolution: forward and data gradient
// ---------------------------------------------------------------------------
// Weight operand of a halo k-block: rows n (output channels in the forward
// pass, input channels in the data gradient); chunk c of the k-block is chunk
// q = kb*CPB + c of the channel block, whose weight column comes from the
// chunk table. Every thread owns the same chunk c = tid % CPB in all its rows.
template <typename T, int ROWS, int BK, int NT = 256>
struct TapRowLoader {
  static constexpr int VEC = TT<T>::VEC, CPB = BK / VEC, LDK = BK + UN_LDS_PAD_CHUNKS * VEC;
  static constexpr int CHUNKS = ROWS * CPB, NV = CHUNKS >= NT ? CHUNKS / NT : 1;
  // fewer chunks than threads: the first CHUNKS threads (whole waves) move them
  static constexpr bool PART = CHUNKS < NT;
  static_assert((CHUNKS % NT == 0 || NT % CHUNKS == 0) && NT % CPB == 0 && CHUNKS % 64 == 0,
                "chunks must spread evenly over whole waves");
  __amdgpu_buffer_rsrc_t rsrc;
  int rowoff[NV];
  u32x4 r[2][NV];  // two k-blocks in flight (register slots 0 and 1)
  __device__ __forceinline__ bool active() const { return !PART || (int)threadIdx.x < CHUNKS; }
  __device__ __forceinline__ void init(const T* base, int64_t ld, int rows_valid) {
    rsrc = make_rsrc(base, (int64_t)rows_valid * ld * (int64_t)sizeof(T));
#pragma unroll
    for (int s = 0; s < NV; ++s) rowoff[s] = (int)((threadIdx.x + NT * s) / CPB) * (int)ld * (int)sizeof(T);
  }
  // col: weight column of this thread's chunk, or -1 for a chunk past the block's end
  template <int S>
  __device__ __forceinline__ void load(int col) {
    if (!active()) return;
#pragma unroll
    for (int s = 0; s < NV; ++s)
      r[S][s] = col < 0 ? zero4()
                        : __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, rowoff[s] + col * (int)sizeof(T), 0, 0));
  }
  template <int S>
  __device__ __forceinline__ void store(T* sm) const {
    if (!active()) return;
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      const int v = threadIdx.x + NT * s;
      *(u32x4*)(sm + (v / CPB) * LDK + (v % CPB) * VEC) = r[S][s];
    }
  }
};

// The elements e = (position, 16-byte chunk) of a staged halo block that one
// thread moves: e = tid, tid + NT, ... The thread steps its (chunk, column,
// row, image) by the uniform decomposition of NT with carries (no per-element
// division; when the chunks per position divide NT, FIX, a thread's chunk
// never changes). Source offsets: the image's base kept as a running sum,
// rows and columns by 24-bit multiplies (rows of under 2^24 elements, tensors
// of under 2^31 bytes). Staged block: LDS [img][hr][hc][cs], channels
// [c0, c0 + cbw) of the source. Forward: the conv input X. Data gradient: dZ,
// expanded from the pooled gradient G and the window argmax.
template <typename T, bool DGRAD, int NT>
struct HaloWalk {
  static constexpr int VEC = TT<T>::VEC;
  int cpp, imgs, hc, hr, dch, dhc, dhr, dimg, dst_step, dst_wrap;
  // source geometry: rows of ROW elements, images of IMG, channel stride CH;
  // position (hrow, hcol) reads row ybase + hrow, column xbase + hcol
  int YL, XL, ROW, CH, ybase, xbase, lastimg, c0;
  unsigned IMG;
  // this thread's element
  int chi, hcol, hrow, img, dst;
  unsigned nb;
  __device__ __forceinline__ HaloWalk(const ConvProb& p, int img0, int y0, int c0_, int cbw, float rc_cpp) {
    const bool pool = DGRAD && p.pool;
    cpp = cbw / VEC;
    imgs = p.imgs;
    hc = p.hc;
    hr = p.hr;
    c0 = c0_;
    const int cs = p.cs, plane = hr * hc, dpos = NT / cpp, dr0 = dpos - (dpos / plane) * plane;
    dch = NT - dpos * cpp;
    dimg = dpos / plane;
    dhr = dr0 / hc;
    dhc = dr0 - dhr * hc;
    dst_step = dpos * cs + dch * VEC;
    dst_wrap = cs - cbw;
    CH = DGRAD ? p.O : p.C;
    YL = DGRAD ? (pool ? 2 * p.PH : p.OH) : p.H;
    XL = DGRAD ? (pool ? 2 * p.PW : p.OW) : p.W;
    ROW = (DGRAD ? (pool ? p.PW : p.OW) : p.W) * CH;
    IMG = (unsigned)(DGRAD ? (pool ? p.PH : p.OH) : p.H) * (unsigned)ROW;
    ybase = DGRAD ? y0 + p.pad - (p.KH - 1) : y0 - p.pad;
    xbase = DGRAD ? p.pad - (p.KH - 1) : -p.pad;
    lastimg = p.Nb - img0;  // images at or past it are past the batch
    int rem;
    const int pos = SmallDiv(cpp, rc_cpp).qr(threadIdx.x, chi);
    img = SmallDiv(plane, p.rc_plane).qr(pos, rem);
    hrow = SmallDiv(hc, p.rc_hc).qr(rem, hcol);
    dst = pos * cs + chi * VEC;
    nb = (unsigned)(img0 + img) * IMG;
  }
  __device__ __forceinline__ bool live() const { return img < imgs; }
  // source element offset of the current element (shift sh: un-pooled rows
  // and columns of a pooled gradient) and whether it lies in the image
  template <int SH>
  __device__ __forceinline__ unsigned src(bool& in, int& y, int& x) const {
    y = ybase + hrow;
    x = xbase + hcol;
    in = img < imgs && img < lastimg && (unsigned)y < (unsigned)YL && (unsigned)x < (unsigned)XL;
    return nb + __umul24((unsigned)(y >> SH), (unsigned)ROW) + __umul24((unsigned)(x >> SH), (unsigned)CH) +
           (unsigned)(c0 + chi * VEC);
  }
  // the next element, NT on
  template <bool FIX>
  __device__ __forceinline__ void next() {
    dst += dst_step;
    hcol += dhc;
    hrow += dhr;
    img += dimg;
    nb += (unsigned)dimg * IMG;
    if constexpr (!FIX) {
      chi += dch;
      if (chi >= cpp) {
        chi -= cpp;
        dst += dst_wrap;
        ++hcol;
      }
    }
    if (hcol >= hc) {
      hcol -= hc;
      ++hrow;
    }
    if (hrow >= hr) {
      hrow -= hr;
      ++img;
      nb += IMG;
    }
  }
};

// Stage channels [c0, c0 + cbw) of the operand rows a halo tile reads into
// LDS, [img][hr][hc][cs]; positions outside the image (padding), past the
// batch, or - data gradient - not receiving the window's gradient are zero.
// Every element is loaded through buffer resources: one outside the image
// reads at an offset past the range, which returns zero.
template <typename T, bool DGRAD, int NT = 256>
__device__ __forceinline__ void stage_halo(const ConvProb& p, T* sH, int img0, int y0, int c0, int cbw, float rc_cpp) {
  // four loads in flight per thread (six or eight measured no faster for
  // the data gradient's larger blocks)
  constexpr int UNR = 4;
  constexpr uint32_t OOB = 0x80000000u;
  HaloWalk<T, DGRAD, NT> w(p, img0, y0, c0, cbw, rc_cpp);
  const bool pool = DGRAD && p.pool;
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(DGRAD ? p.G : p.X, (int64_t)p.Nb * w.IMG * (int64_t)sizeof(T));
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(p.gam, pool ? (int64_t)p.Nb * w.IMG : 0);
  auto run = [&](auto fixed_chunk, auto shift) {
    constexpr bool FIX = decltype(fixed_chunk)::value;
    constexpr int SH = decltype(shift)::value;
    while (w.live()) {
      u32x4 v[UNR];
      int dd[UNR];
#pragma unroll
      for (int k = 0; k < UNR; ++k) {
        dd[k] = w.live() ? w.dst : -1;
        bool in;
        int y, x;
        const unsigned off = w.template src<SH>(in, y, x);
        v[k] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, in ? off * (unsigned)sizeof(T) : OOB, 0, 0));
        if (SH) select_am<T>(v[k], load_am_buf<T>(ra, in ? off : OOB), ((y & 1) << 1) | (x & 1));
        w.template next<FIX>();
      }
#pragma unroll
      for (int k = 0; k < UNR; ++k)
        if (dd[k] >= 0) *(u32x4*)(sH + dd[k]) = v[k];
    }
  };
  using F = std::false_type;
  using Tr = std::true_type;
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  if (pool) {
    if (w.dch == 0) run(Tr{}, S1{});
    else run(F{}, S1{});
  } else {
    if (w.dch == 0) run(Tr{}, S0{});
    else run(F{}, S0{});
  }
}

// The forward halo block of a tile (origin img0, y0), loaded into registers
// only: this thread's first PF elements, v[k] bound for LDS element dd[k]
// (-1: none). Multi-tile workgroups fetch the next tile's rows this way before
// the current tile's epilogue stores (loads and stores share one in-order
// counter), and write them to LDS after it (put_halo); the host enables them
// only where PF elements per thread cover the block.
template <typename T, int NT, int PF>
__device__ __forceinline__ void fetch_halo(const ConvProb& p, int img0, int y0, float rc_cpp, u32x4 (&v)[PF],
                                           int (&dd)[PF]) {
  constexpr uint32_t OOB = 0x80000000u;
  HaloWalk<T, false, NT> w(p, img0, y0, 0, p.C, rc_cpp);
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(p.X, (int64_t)p.Nb * w.IMG * (int64_t)sizeof(T));
#pragma unroll
  for (int k = 0; k < PF; ++k) {
    dd[k] = w.live() ? w.dst : -1;
    bool in;
    int y, x;
    const unsigned off = w.template src<0>(in, y, x);
    v[k] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, in ? off * (unsigned)sizeof(T) : OOB, 0, 0));
    w.template next<false>();
  }
}
template <typename T, int PF>
__device__ __forceinline__ void put_halo(T* sH, const u32x4 (&v)[PF], const int (&dd)[PF]) {
#pragma unroll
  for (int k = 0; k < PF; ++k)
    if (dd[k] >= 0) *(u32x4*)(sH + dd[k]) = v[k];
}

// One k-block of a halo tile: A rows read from the staged halo at the lane's
// row base plus the chunk's tap offset, B from the weight stage. Chunks at or
// past nq have zero weights.
// bf16: 32x32x16 MFMA blocks (Acc32); a k-step of 16 spans two chunks, lane
// half h = lane / 32 supplying chunk qs + h. Row bases and tap offsets are in
// bytes; the offsets of k-block kb are laid out as qa[8 kb + 4 h + s] = the
// offset of chunk 8 kb + 2 s + h (clamped to the last chunk), so a lane reads
// the four it needs at once.
template <int BM, int BN, int BK, int NW>
__device__ __forceinline__ void mma_halo(const bf16_t* sH, const int (&hbase)[Acc32<BM, BN, NW>::FM], const int* qa,
                                         int q0, int nq, const bf16_t* sB, typename Acc32<BM, BN, NW>::Acc& acc) {
  using L = Acc32<BM, BN, NW>;
  constexpr int LDK = Tile<bf16_t, BM, BN, BK, NW>::LDK;
  static_assert(BK == 64, "eight chunks per k-block, four k-steps");
  const int lane = threadIdx.x & 63, h = lane >> 5;
  const char* hp[L::FM];
#pragma unroll
  for (int i = 0; i < L::FM; ++i) hp[i] = (const char*)sH + hbase[i];
  const bf16_t* sb = sB + (L::wave_n() + (lane & 31)) * LDK + 8 * h;
  const u32x4 t = *(const u32x4*)(qa + q0 + 4 * h);
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    if (q0 + 2 * s < nq) {
      const int ao = (int)t[s];
      const bf16x8 b = __builtin_bit_cast(bf16x8, *(const u32x4*)(sb + 16 * s));
#pragma unroll
      for (int i = 0; i < L::FM; ++i) {
        const bf16x8 a = __builtin_bit_cast(bf16x8, *(const u32x4*)(hp[i] + ao));
        acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[i], 0, 0, 0);
      }
    }
  }
}

// fp32: 16x16x4 MFMA blocks (Acc16).
template <int BM, int BN, int BK, int NW>
__device__ __forceinline__ void mma_halo(const float* sH, const int (&hbase)[Acc16<float, BM, BN, BK, NW>::FM],
                                         const int* qa, int q0, int nq, const float* sB,
                                         typename Acc16<float, BM, BN, BK, NW>::Acc& acc) {
  using TL = Tile<float, BM, BN, BK, NW>;
  constexpr int VEC = TT<float>::VEC;
  const int lane = threadIdx.x & 63;
  const int wn = TL::wave_n();
  const int lr = lane & 15, lg = lane >> 4;
#pragma unroll
  for (int kk = 0; kk < BK; kk += 16) {
    const int qs = q0 + kk / VEC;
    if (qs < nq) {
      const int ao = qa[min(qs + lg, nq - 1)];
      f32x4 a[TL::FM], b[TL::FN];
#pragma unroll
      for (int i = 0; i < TL::FM; ++i) a[i] = *(const f32x4*)(sH + hbase[i] + ao);
#pragma unroll
      for (int j = 0; j < TL::FN; ++j) b[j] = *(const f32x4*)(sB + (wn + 16 * j + lr) * TL::LDK + kk + 4 * lg);
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int i = 0; i < TL::FM; ++i)
#pragma unroll
          for (int j = 0; j < TL::FN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][q], b[j][q], acc[i][j], 0, 0, 0);
    }
  }
}

// LDS of a halo tile: [weight stages][qa][qb][staged rows], halo_elems() of them.
template <typename T, int BN, int BK>
struct HaloSmem {
  static constexpr int B_ELEMS = BN * (BK + 16 / (int)sizeof(T));
  static constexpr int HALO = halo_elems(sizeof(T), BN, BK);
  static constexpr size_t BYTES = (2 * (size_t)B_ELEMS + HALO) * sizeof(T) + 2 * HALO_QMAX * sizeof(int);
};

// The BM x BN halo tile `local` of problem p and, for a multi-tile forward
// workgroup (p.mt > 1: one channel block), the next p.mt - 1 m-tiles of the
// same n-column. Those reuse the tap tables and row bases, and (at most two
// k-blocks) the weights in LDS; their rows are fetched into registers before
// the previous tile's epilogue.
template <typename T, int BM, int BN, int BK, bool DGRAD, int NW>
__device__ __forceinline__ void halo_tile(const ConvProb& p, int local, char* smem) {
  using TL = Tile<T, BM, BN, BK, NW>;
  using L = std::conditional_t<sizeof(T) == 2, Acc32<BM, BN, NW>, Acc16<T, BM, BN, BK, NW>>;
  constexpr int NT = TL::NT;
  using HS = HaloSmem<T, BN, BK>;
  constexpr int VEC = TT<T>::VEC, CPB = BK / VEC;
  static_assert(TL::B_ELEMS == HS::B_ELEMS, "halo LDS budget assumes one pad chunk per row");
  static_assert(NT == (sizeof(T) == 2 ? HALO_NT_BF16 : HALO_NT_F32), "halo workgroup size");
  T* sB = (T*)smem;
  int* qa = (int*)(sB + 2 * TL::B_ELEMS);
  int* qb = qa + HALO_QMAX;
  T* sH = (T*)(qb + HALO_QMAX);
  const int tm0 = local / p.tiles_n, tn = local - tm0 * p.tiles_n;
  const int n0 = tn * BN;
  const int SH = DGRAD ? p.H : p.OH, SW = DGRAD ? p.W : p.OW;
  // (not the tall tiles: their accumulators leave no registers for the
  // fetched rows across the epilogue; the host plans none)
  constexpr bool MULTI = !DGRAD && BM <= 2 * (sizeof(T) == 2 ? CONV_BM_BF16 : CONV_BM_F32);
  const int mt = MULTI ? max(1, min(p.mt, p.tiles_m - tm0)) : 1;
  // first operand image and row of m-tile tm
  auto origin = [&](int tm, int& img0, int& y0) {
    if (p.imgs > 1) {
      img0 = tm * p.imgs;
      y0 = 0;
    } else {
      const int tpi = SH / p.tr;
      img0 = tm / tpi;
      y0 = (tm - img0 * tpi) * p.tr;
    }
  };
  int img0, y0;
  origin(tm0, img0, y0);
  // halo offset of the first tap of each of this lane's MFMA rows
  int hbase[L::FM];
  {
    const bool wo = !DGRAD && p.pool;  // window order: r = 4 * window + (dy, dx)
    const int per_row = wo ? SW >> 1 : SW, per_img = wo ? (p.tr >> 1) * per_row : p.tr * SW;
    const SmallDiv dimg(per_img, p.rc_img), drow(per_row, p.rc_row);
    const int hr = p.hr, hc = p.hc, cs = p.cs;
#pragma unroll
    for (int i = 0; i < L::FM; ++i) {
      const int r = L::arow(i), u = wo ? r >> 2 : r, d = r & 3;
      int rem, col;
      const int img = dimg.qr(u, rem), row = drow.qr(rem, col);
      const int y = wo ? 2 * row + (d >> 1) : row, x = wo ? 2 * col + (d & 1) : col;
      hbase[i] = ((img * hr + y) * hc + x) * cs * (sizeof(T) == 2 ? 2 : 1);  // bf16: bytes
    }
  }

  typename L::Acc acc;
  L::zero(acc);

  TapRowLoader<T, BN, BK, NT> lb;
  lb.init((const T*)p.Wt + (int64_t)n0 * p.ldw, p.ldw, p.N - n0);
  const int KH = p.KH, Cin = DGRAD ? p.O : p.C, cq = threadIdx.x % CPB, hc = p.hc, cs = p.cs;
  const SmallDiv dkh(KH, p.rc_kh);
  // weight column of chunk q of the channel block at c0 (cpt chunks per tap;
  // -1 past its nq chunks)
  auto col_of = [&](int q, const SmallDiv& dcpt, int nq, int c0) {
    int cr;
    const int tap = dcpt.qr(q, cr);
    return q < nq ? tap * Cin + c0 + cr * VEC : -1;
  };
  // the k loop of a channel block of nq chunks (nkb k-blocks), whose first
  // k-block is in LDS buffer 0 and second in register slot 1. Iteration kb
  // (P = kb & 1): load k-block kb + 2 into slot P (its k-block kb is in LDS
  // already), run k-block kb from LDS buffer P, move k-block kb + 1 from slot
  // P ^ 1 to LDS buffer P ^ 1 (last read in iteration kb - 1)
  auto kloop = [&](int nq, int nkb) {
    auto step = [&](auto par, int kb) {
      constexpr int P = decltype(par)::value;
      if (kb + 2 < nkb) {
        const int q = (kb + 2) * CPB + cq;
        lb.template load<P>(q < nq ? qb[q] : -1);
      }
      mma_halo<BM, BN, BK, NW>(sH, hbase, qa, kb * CPB, nq, sB + P * TL::B_ELEMS, acc);
      if (kb + 1 < nkb) lb.template store<P ^ 1>(sB + (P ^ 1) * TL::B_ELEMS);
      __syncthreads();
    };
    int kb = 0;
    for (; kb + 1 < nkb; kb += 2) {
      step(std::integral_constant<int, 0>{}, kb);
      step(std::integral_constant<int, 1>{}, kb + 1);
    }
    if (kb < nkb) step(std::integral_constant<int, 0>{}, kb);
  };
  for (int c0 = 0; c0 < Cin; c0 += p.cb) {
    const int cbw = min(p.cb, Cin - c0), cpt = cbw / VEC, nq = KH * KH * cpt;
    const SmallDiv dcpt(cpt, c0 + p.cb >= Cin ? p.rc_cpt_last : p.rc_cpt);
    // the weights of k-blocks 0 and 1 first (columns computed directly), so
    // their loads overlap the staging of the operand rows; k-block kb sits in
    // register slot kb & 1 and LDS buffer kb & 1
    lb.template load<0>(col_of(cq, dcpt, nq, c0));
    lb.template load<1>(col_of(CPB + cq, dcpt, nq, c0));
    __syncthreads();  // the previous channel block's halo, tables and weight stages are no longer read
    // qa: the halo offset of a chunk's tap and channels (bf16: in bytes, in
    // the k-block layout of mma_halo, padded to whole k-blocks); qb: its
    // weight column (fwd: W[o][(tap, c)]; dgrad: WT[c][(tap, o)])
    auto tap_off = [&](int q, int& col) {
      int cr, v;
      const int tap = dcpt.qr(q, cr), ch = cr * VEC, u = dkh.qr(tap, v);
      col = tap * Cin + c0 + ch;
      return (DGRAD ? (KH - 1 - u) * hc + (KH - 1 - v) : u * hc + v) * cs + ch;
    };
    if constexpr (sizeof(T) == 2) {
      static_assert(CPB == 8, "bf16 table layout");
      const int nqa = (nq + 7) & ~7;
      for (int e = threadIdx.x; e < nqa; e += NT) {
        int col;
        qa[e] = 2 * tap_off(min((e & ~7) + 2 * (e & 3) + ((e >> 2) & 1), nq - 1), col);
        if (e < nq) {
          tap_off(e, col);
          qb[e] = col;
        }
      }
    } else {
      for (int q = threadIdx.x; q < nq; q += NT) {
        int col;
        qa[q] = tap_off(q, col);
        qb[q] = col;
      }
    }
    stage_halo<T, DGRAD, NT>(p, sH, img0, y0, c0, cbw, dcpt.r);
    lb.template store<0>(sB);
    __syncthreads();
    kloop(nq, (nq + CPB - 1) / CPB);
  }
  if constexpr (DGRAD) {
    conv_dgrad_epilogue<T, BM, BN, L>(p, tm0 * BM, n0, acc, smem);
  } else {
    // the epilogue, then any further m-tiles (mt > 1: one channel block, whose
    // tables stay in LDS). The k loop's last barrier has freed the staged
    // rows; at most two k-blocks leave both weight buffers (and register slot
    // 1) as they are.
    const int cpt = Cin / VEC, nq = KH * KH * cpt, nkb = (nq + CPB - 1) / CPB;
    const SmallDiv dcpt(cpt, p.rc_cpt_last);
    for (int t = 1;; ++t) {
      const bool more = MULTI && t < mt;
      u32x4 hv[HALO_PF];
      int hd[HALO_PF];
      if (more) {
        int nimg0, ny0;
        origin(tm0 + t, nimg0, ny0);
        fetch_halo<T, NT, HALO_PF>(p, nimg0, ny0, dcpt.r, hv, hd);
        if (nkb > 2) {
          lb.template load<0>(col_of(cq, dcpt, nq, 0));
          lb.template load<1>(col_of(CPB + cq, dcpt, nq, 0));
        }
      }
      conv_fwd_epilogue<T, L>(p, (tm0 + t - 1) * BM, n0, acc);
      if (!more) break;
      L::zero(acc);
      put_halo<T, HALO_PF>(sH, hv, hd);
      if (nkb > 2) lb.template store<0>(sB);
      __syncthreads();
      kloop(nq, nkb);
    }
  }
}

// Halo-tiled conv pass; each problem's tile shape (p.bm x p.bn) is the wide
// BM x BN, the narrow 2BM x BN/2 or (bf16 forward only) the tall 4BM x BN/2 one,
// so a launch mixes them. LDS is dynamic, sized
// by the host for the launch's largest staged block (small halos leave room
// for more workgroups per CU).
// Waves of a halo workgroup (bf16; fp32 keeps 4): a 4-wave workgroup runs
// three per CU, larger ones two.
template <typename T> constexpr int halo_waves() { return sizeof(T) == 2 ? UN_HALO_WAVES : 4; }
template <typename T> constexpr int halo_wpe() { return halo_waves<T>() == 4 ? 3 : halo_waves<T>() / 2; }

template <typename T, int BM, int BN, int BK, bool DGRAD>
__global__ __launch_bounds__((64 * halo_waves<T>())) __attribute__((amdgpu_waves_per_eu((halo_wpe<T>()))))
void conv_halo_kernel(const ConvProb* __restrict__ probs, const int32_t* __restrict__ tile_map) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int prob = tile_map[2 * blockIdx.x], local = tile_map[2 * blockIdx.x + 1];
  if (prob < 0) return;  // padding of the XCD-ordered tile list
  const ConvProb& p = probs[prob];
  constexpr int NW = halo_waves<T>();
  if (p.bn == BN) {
    halo_tile<T, BM, BN, BK, DGRAD, NW>(p, local, smem);
  } else if (DGRAD || sizeof(T) != 2 || p.bm == 2 * BM) {
    halo_tile<T, 2 * BM, BN / 2, BK, DGRAD, NW>(p, local, smem);
  } else {
    if constexpr (!DGRAD && sizeof(T) == 2) halo_tile<T, 4 * BM, BN / 2, BK, DGRAD, NW>(p, local, smem);
  }
}

template <typename T, int BM, int BN, int BK, int MODE>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void conv_wgrad_kernel(const ConvProb* __restrict__ probs,
                                                         const int32_t* __restrict__ tile_map, int64_t wsoff) {
  using TL = Tile<T, BM, BN, BK>;
  __shared__ __attribute__((aligned(16))) char smem[Smem<T, BM, BN, BK>::BYTES];
  const int prob = tile_map[2 * blockIdx.x];
  int local = tile_map[2 * blockIdx.x + 1];
  if (prob < 0) return;  // padding of the XCD-ordered tile list
  const ConvProb& p = probs[prob];
  const int per_split = p.tiles_m * p.tiles_n;
  const int split = local / per_split;
  local -= split * per_split;
  const int tm = local / p.tiles_n, tn = local - tm * p.tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;

  f32x4 acc[TL::FM][TL::FN];
#pragma unroll
  for (int i = 0; i < TL::FM; ++i)
#pragma unroll
    for (int j = 0; j < TL::FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  WgradLoader<T, BM, BN, BK, MODE> ld;
  ld.init(p, m0, n0);
  const int nkb = (p.K + BK - 1) / BK;
  const int kb0 = split * p.kchunk, kb1 = min(nkb, kb0 + p.kchunk);
  mma_loop1<T, BM, BN, BK>(ld, kb0, kb1, (T*)smem, acc);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = (wave >> 1) * TL::WM, wn = (wave & 1) * TL::WN;
  float* ws = (float*)((char*)p.ws + wsoff) + (int64_t)split * p.O * p.ldws;
#pragma unroll
  for (int i = 0; i < TL::FM; ++i) {
    const int mb = m0 + wm + 16 * i + 4 * (lane >> 4);
    if (mb >= p.M) continue;
    const int nv = min(4, p.M - mb);
#pragma unroll
    for (int j = 0; j < TL::FN; ++j) {
      const int n = n0 + wn + 16 * j + (lane & 15);
      if (n >= p.N) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (r < nv) ws[(int64_t)(mb + r) * p.ldws + n] = acc[i][j][r];
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 conv weight gradient on the grouped GEMM's machinery: 16 waves of
// 32x32x16 MFMA tiles, loads two k-blocks ahead, and both operands staged in
// LDS k-major - as they lie in memory, [pixel][channel] - and turned into MFMA
// operands by the LDS transpose reads. For blocks whose channel counts O and
// C are whole 16-byte vectors (pooled or not).
//   A (rows o):      dZ[pixel][o], gathered from the pooled gradient G[w][o]
//                    and the window argmax (pooled), or G[pixel][o] itself;
//   B (rows j):      the input patch X[n][y+u-pad][x+v-pad][c], j = (u,v,c),
//                    and the bias column j == KH*KW*C reading 1.
// Each thread moves one 16-byte chunk of each operand per k-block: pixel
// k = t / CPR of the block, rows 8*(t % CPR) .. +7. Pixels of a pooled block
// are ordered m = 4*w + (dy*2 + dx), so k % 4 is the window position.
// The k-loop is bound by vector-instruction issue, not by the MFMA units:
// the loaders keep their addresses as running offsets and the operand pixel
// coordinates as counters stepped once per k-block (uniform steps, carries by
// compare and subtract), with no per-block division or 32-bit multiply (both
// quarter-rate). Offsets are 32-bit: every conv tensor is under 2^31 bytes.
template <int ROWS, int BK, int NT, int SLOTS, int PAD, bool POOL>
struct ConvKA {
  static constexpr int VEC = 8, CPR = ROWS / VEC, LDR = ROWS + PAD, NV = BK * CPR / NT;
  static_assert(NV >= 1 && BK * CPR == NV * NT, "whole chunks per thread and k-block");
  static_assert(BK % 4 == 0 && (NT / CPR) % 4 == 0, "k-blocks hold whole windows; a thread's chunks share one window position");
  __amdgpu_buffer_rsrc_t rs, rs_am;
  uint32_t offb, offa, stepb, stepa;  // byte offsets of chunk 0 in G and in the argmax bytes, and their steps
  uint32_t sb1, sa1;                  // from chunk s to chunk s + 1 (NT / CPR pixels on)
  int sm_off;
  u32x4 r[SLOTS][NV];
  uint64_t am[SLOTS][NV];
  // Chunk s of a thread: pixel k + s * (NT / CPR) of the block. Channels
  // o >= O are read without a range test: they feed accumulator rows that
  // are never stored. Pixels past the last one lie past both buffers' ranges
  // and read zero.
  __device__ __forceinline__ void init(const ConvProb& p, int o0, int kb0) {
    const int k = threadIdx.x / CPR, o = o0 + (threadIdx.x % CPR) * VEC;
    const int pix = kb0 * BK + k;
    const uint32_t e = (uint32_t)((POOL ? pix >> 2 : pix) * p.O + o);  // element offset of chunk 0 in G
    const uint32_t step = (uint32_t)((POOL ? BK / 4 : BK) * p.O), s1 = (uint32_t)((POOL ? NT / CPR / 4 : NT / CPR) * p.O);
    offb = 2 * e;
    offa = e;
    stepb = 2 * step;
    stepa = step;
    sb1 = 2 * s1;
    sa1 = s1;
    sm_off = kmaj_bf16<LDR>(k, (threadIdx.x % CPR) * VEC);
    const int64_t rows = POOL ? (int64_t)p.Nb * p.PH * p.PW : (int64_t)p.Nb * p.OH * p.OW;
    rs = make_rsrc(p.G, rows * p.O * (int64_t)sizeof(bf16_t));
    if constexpr (POOL) rs_am = make_rsrc(p.gam, rows * p.O);
  }
  // the next k-block (the loop issues blocks in order, one call each)
  template <int S>
  __device__ __forceinline__ void load(int) {
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      r[S][s] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, offb + s * sb1, 0, 0));
      if constexpr (POOL) am[S][s] = load_am_buf<bf16_t>(rs_am, offa + s * sa1);
    }
    offb += stepb;
    offa += stepa;
  }
  template <int S>
  __device__ __forceinline__ void store(bf16_t* sm) const {
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      u32x4 v = r[S][s];
      if constexpr (POOL) select_am<bf16_t>(v, am[S][s], (threadIdx.x / CPR) & 3);
      *(u32x4*)(sm + sm_off + (s * (NT / CPR)) * LDR) = v;
    }
  }
};

// Chunk s of a thread: output pixel k + s * (NT / CPR) of the block, input
// position (n, y + u - pad, x + v - pad) of the chunk's tap (u, v), with
// y = F*a + dy, x = F*b + dx: (a, b) is a pooled block's window (pixel order
// 4 * window + (dy, dx)), else the pixel itself (F = 1, dy = dx = 0). Pixels
// past the last one have n >= Nb: their input rows lie past the buffer's range
// and read zero (the gradient operand is zero there too). The bias column
// J reads ones; columns past it feed output columns that are never stored.
//
// Every k-block moves a chunk by BK pixels. UNI: the k-blocks are whole rows
// of windows within one image, or whole images, so every lane moves by the
// same rows and the wrap to the next image is the same for all: a lane keeps
// its input row and byte offset, stepped by wave-uniform amounts. Otherwise a
// lane keeps (a, b) and the element offset q and wraps them itself.
template <int ROWS, int BK, int NT, int SLOTS, int PAD, bool POOL, bool UNI>
struct ConvKB {
  static constexpr int VEC = 8, CPR = ROWS / VEC, LDR = ROWS + PAD, NV = BK * CPR / NT, F = POOL ? 2 : 1;
  static constexpr int ST = POOL ? BK / 4 : BK;  // windows (or pixels) per k-block
  static constexpr uint32_t OOB = 0x7ffffff0u;   // a byte offset past every range: the load returns zero
  static_assert(NV >= 1 && BK * CPR == NV * NT, "whole chunks per thread and k-block");
  static_assert(NT % CPR == 0 && (NT / CPR) % 4 == 0, "a thread's chunks share one row set and window position");
  __device__ __forceinline__ static bool uniform(const ConvProb& pr) {
    const int A = POOL ? pr.PH : pr.OH, B = POOL ? pr.PW : pr.OW, plane = A * B;
    return (ST % B == 0 && plane % ST == 0) || ST % plane == 0;
  }
  __amdgpu_buffer_rsrc_t rs;
  int H, W, A, B, ey, ex, sm_off;
  uint32_t orm;  // ORed into the first word: the bias column's 1.0, else 0
  bool jin;
  // general stepping
  int sa, sb, q0, q1, q2;
  int a[NV], b[NV], q[NV];
  // uniform stepping: the block's first window row ablk, rows per block ra,
  // and the row / byte steps of a block without (n) and with (w) the wrap
  int ablk, ra, dyn, dyw;
  uint32_t dqn, dqw;
  int iy[NV];
  uint32_t qb[NV];
  bool xin[NV];
  u32x4 r[SLOTS][NV];
  __device__ __forceinline__ void init(const ConvProb& pr, int j0, int kb0) {
    const int k = threadIdx.x / CPR;
    const int j = j0 + (threadIdx.x % CPR) * VEC, J = pr.KH * pr.KH * pr.C;
    jin = j < J;
    orm = j == J ? bits_of<bf16_t>(TT<bf16_t>::from_f(1.0f)) : 0u;
    const int tap = j / pr.C, c0 = j - tap * pr.C, u = tap / pr.KH, v = tap - u * pr.KH;
    H = pr.H;
    W = pr.W;
    A = POOL ? pr.PH : pr.OH;
    B = POOL ? pr.PW : pr.OW;
    const int d = POOL ? (k & 3) : 0, dy = d >> 1, dx = d & 1;
    ey = dy + u - pr.pad;  // input row of the chunk's pixel: F * a + ey
    ex = dx + v - pr.pad;
    sm_off = kmaj_bf16<LDR>(k, (threadIdx.x % CPR) * VEC);
    const int plane = A * B;
    if constexpr (UNI) {
      const int C2 = 2 * pr.C;
      if (ST % plane == 0) {  // whole images per block
        ra = 0;
        dyn = dyw = 0;
        dqn = dqw = (uint32_t)((ST / plane) * H * W * C2);
      } else {  // whole rows of one image per block
        ra = ST / B;
        dyn = F * ra;
        dyw = F * ra - F * A;
        dqn = (uint32_t)(F * ra * W * C2);
        dqw = (uint32_t)((F * ra * W + H * W - F * A * W) * C2);
      }
      ablk = ((kb0 * ST) % plane) / B;
    } else {
      // the step of BK pixels (BK / 4 windows) in (n, a, b) and its offsets
      const int sn = ST / plane, rem = ST - sn * plane;
      sa = rem / B;
      sb = rem - sa * B;
      q0 = (sn * H * W + F * sa * W + F * sb) * pr.C;  // every step
      q1 = (F * W - F * B) * pr.C;                      // b wrapped: next row of windows
      q2 = (H * W - F * A * W) * pr.C;                  // a wrapped: next image
    }
#pragma unroll
    for (int s = 0; s < NV; ++s) {
      const int pix = kb0 * BK + k + s * (NT / CPR), m = POOL ? pix >> 2 : pix;
      const int n = m / plane, r2 = m - n * plane;
      const int aa = r2 / B, bb = r2 - aa * B;
      if constexpr (UNI) {
        iy[s] = F * aa + ey;
        const int ix = F * bb + ex;
        xin[s] = jin && (unsigned)ix < (unsigned)W;
        // modulo 2^32: exact again once the row is inside the image
        qb[s] = 2u * (uint32_t)(((n * H + iy[s]) * W + ix) * pr.C + c0);
      } else {
        a[s] = aa;
        b[s] = bb;
        q[s] = ((n * H + F * aa + ey) * W + F * bb + ex) * pr.C + c0;
      }
    }
    rs = make_rsrc(pr.X, (int64_t)pr.Nb * pr.H * pr.W * pr.C * (int64_t)sizeof(bf16_t));
  }
  // the next k-block (the loop issues blocks in order, one call each)
  template <int S>
  __device__ __forceinline__ void load(int) {
    if constexpr (UNI) {
      int dy = dyn;
      uint32_t dq = dqn;
      ablk += ra;
      if (ablk >= A) {  // wave-uniform: the next block starts the next image
        ablk -= A;
        dy = dyw;
        dq = dqw;
      }
#pragma unroll
      for (int s = 0; s < NV; ++s) {
        const bool in = xin[s] && (unsigned)iy[s] < (unsigned)H;
        u32x4 val = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, in ? qb[s] : OOB, 0, 0));
        val[0] |= orm;
        r[S][s] = val;
        iy[s] += dy;
        qb[s] += dq;
      }
    } else {
#pragma unroll
      for (int s = 0; s < NV; ++s) {
        const int iyy = F * a[s] + ey, ix = F * b[s] + ex;
        const bool in = jin && (unsigned)iyy < (unsigned)H && (unsigned)ix < (unsigned)W;
        u32x4 val = __builtin_bit_cast(
            u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, in ? (uint32_t)q[s] * 2u : OOB, 0, 0));
        val[0] |= orm;
        r[S][s] = val;
        q[s] += q0;
        b[s] += sb;
        const bool cb = b[s] >= B;
        b[s] -= cb ? B : 0;
        q[s] += cb ? q1 : 0;
        a[s] += sa + (cb ? 1 : 0);
        const bool ca = a[s] >= A;
        a[s] -= ca ? A : 0;
        q[s] += ca ? q2 : 0;
      }
    }
  }
  template <int S>
  __device__ __forceinline__ void store(bf16_t* sm) const {
#pragma unroll
    for (int s = 0; s < NV; ++s) *(u32x4*)(sm + sm_off + (s * (NT / CPR)) * LDR) = r[S][s];
  }
};

// NARROW: tiles of CONV_WG_NARROW_BM output channels (8 waves), for launches
// whose blocks have at most that many; else 128 rows (16 waves).
template <bool POOL, bool NARROW>
__global__ __launch_bounds__((NARROW ? 512 : 1024)) __attribute__((amdgpu_waves_per_eu((NARROW ? 4 : 8))))
void conv_wgrad_mfma_kernel(const ConvProb* __restrict__ probs, const int32_t* __restrict__ tile_map,
                            int64_t wsoff) {
  constexpr int BM = NARROW ? CONV_WG_NARROW_BM : CONV_BM_BF16, BN = CONV_BN_BF16, BK = CONV_BK_BF16;
  using MM = GemmMma<bf16_t, BM, BN, BK, NARROW ? 2 : 4, 4>;  // 32x32 wave tiles
  static_assert(MM::NT == (NARROW ? 512 : 1024), "launch bounds");
  constexpr int NT = MM::NT, D = UN_GEMM_DEPTH;
  static_assert(MM::LDR_A * BK <= Tile<bf16_t, BM, BN, BK>::A_ELEMS &&
                    MM::LDR_B * BK <= Tile<bf16_t, BM, BN, BK>::B_ELEMS, "k-major stages fit the stage buffers");
  __shared__ __attribute__((aligned(16))) char smem[Smem<bf16_t, BM, BN, BK>::BYTES];
  const int prob = tile_map[2 * blockIdx.x];
  int local = tile_map[2 * blockIdx.x + 1];
  if (prob < 0) return;  // padding of the XCD-ordered tile list
  const ConvProb& p = probs[prob];
  const int per_split = p.tiles_m * p.tiles_n;
  const int split = local / per_split;
  local -= split * per_split;
  const int tm = local / p.tiles_n, tn = local - tm * p.tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;
  const int kb0 = split * p.kchunk, nkb = min((p.K + BK - 1) / BK, kb0 + p.kchunk) - kb0;

  typename MM::Acc acc;
  MM::zero(acc);
  ConvKA<BM, BK, NT, D, KMAJ_PAD_BF16, POOL> la;
  la.init(p, m0, kb0);
  using KBU = ConvKB<BN, BK, NT, D, KMAJ_PAD_BF16, POOL, true>;
  if (KBU::uniform(p)) {
    KBU lb;
    lb.init(p, n0, kb0);
    gemm_loop<bf16_t, BM, BN, BK, D, MM, OP_KMAJ, OP_KMAJ>(la, lb, nkb, (bf16_t*)smem, acc);
  } else {
    ConvKB<BN, BK, NT, D, KMAJ_PAD_BF16, POOL, false> lb;
    lb.init(p, n0, kb0);
    gemm_loop<bf16_t, BM, BN, BK, D, MM, OP_KMAJ, OP_KMAJ>(la, lb, nkb, (bf16_t*)smem, acc);
  }

  // this split's partial sums to ws[split][o][j] (32-bit offsets within the
  // split's block of partials)
  const gptr<float> ws = G((float*)((char*)p.ws + wsoff) + (int64_t)split * p.O * p.ldws);
  const int M = p.M, N = p.N, ldws = (int)p.ldws;
  MM::for_groups(acc, [&](int rl, int cl, float (&v)[4]) {
    const int mb = m0 + rl, n = n0 + cl;
    if (n >= N) return;
    const int o = mb * ldws + n;
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (mb + r < M) ws[o + r * ldws] = v[r];
  });
}

// Sum the split-K partials in split order, then the fused SGD update.
template <typename T>
__global__ __launch_bounds__(REDUCE_BLOCK) void reduce_kernel(const ReduceProb* __restrict__ probs,
                                                              const int32_t* __restrict__ blk_prob, float lr,
                                                              const float* __restrict__ lrv,
                                                              const OptHp* __restrict__ opt, int keep_grads,
                                                              int64_t wsoff) {
  const ReduceProb& p = probs[blk_prob[blockIdx.x]];
  const gptr<const float> ws = G((const float*)((const char*)p.ws + wsoff));
  if (lrv) lr = lrv[p.model];
  // 32-bit element indices: a problem's partials are far below 2^31 floats
  const int e = (blockIdx.x - p.blk_base) * REDUCE_BLOCK + threadIdx.x;
  const int J1 = p.J + 1, splits = p.splits, ldws = (int)p.ldws;
  if (e >= p.O * J1) return;
  const int o = (int)((unsigned)e / (unsigned)J1), j = e - o * J1;
  // the sum in split order, eight loads in flight ahead of their adds
  float s = 0.f;
  const int col = o * ldws + j, sstride = p.O * ldws;
  int k = 0;
  for (; k + 8 <= splits; k += 8) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = ws[col + (k + u) * sstride];
#pragma unroll
    for (int u = 0; u < 8; ++u) s += v[u];
  }
  if (k < splits) {
    // the last (splits - k < 8) partials: loads issued together, then added
    // in split order
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = k + u < splits ? ws[col + (k + u) * sstride] : 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (k + u < splits) s += v[u];
  }
  if (j < p.J) {
    const int idx = o * (int)p.ldgw + j;
    if (keep_grads) p.gW[idx] = s;
    // master weight and its copies: touched once per step (non-temporal)
    const float w0 = __builtin_nontemporal_load(G(p.W + idx));
    const float w = opt ? opt_update1(opt[p.model], s, w0, p.s1 + idx, p.s2 + idx) : fmaf(-lr, s, w0);
    __builtin_nontemporal_store(w, G(p.W + idx));
    if (p.Wb) __builtin_nontemporal_store(f2bf(w), G((bf16_t*)p.Wb + idx));
    if (p.WT) {
      const int tap = (int)((unsigned)j / (unsigned)p.C), c = j - tap * p.C;
      G((T*)p.WT)[c * (int)p.ldwt + tap * p.O + o] = TT<T>::from_f(w);
    }
  } else {
    if (keep_grads) p.gb[o] = s;
    p.bmaster[o] = opt ? opt_update1(opt[p.model], s, p.bmaster[o], p.sb1 + o, p.sb2 + o) : fmaf(-lr, s, p.bmaster[o]);
  }
}

// ---------------------------------------------------------------------------
// Softmax cross-entropy, one workgroup per model.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// CE_LANES lanes per sample row (CE_ROWS rows per block, blockIdx.y = model),
// classes strided over the row's lanes; max and sum over the row by a fixed
// butterfly of lane shuffles. dz = (softmax - onehot)/B goes to G. Each
// block sums its rows' losses in row order into partial[model][chunk];
// ce_finish_kernel adds the chunks in order. The grid covers the largest
// batch; a model's blocks beyond its own batch exit.
template <typename T>
__global__ __launch_bounds__(CE_ROWS * CE_LANES) void ce_rows_kernel(const CeProb* __restrict__ probs,
                                                                     const int32_t* __restrict__ labels,
                                                                     int per_model_labels,
                                                                     float* __restrict__ partial, int pstride,
                                                                     int64_t wsoff) {
  __shared__ float rowloss[CE_ROWS];
  const CeProb& p = probs[blockIdx.y];
  const int B = p.B;
  if ((int)blockIdx.x * CE_ROWS >= B) return;  // uniform over the block
  const int32_t* y = labels + (per_model_labels ? p.lab_own : p.lab_shared);
  const int rl = threadIdx.x / CE_LANES, sub = threadIdx.x % CE_LANES;
  const int b = blockIdx.x * CE_ROWS + rl;
  const int C = p.C;
  const bool valid = b < B;
  float* zw = (float*)p.logits + (int64_t)(valid ? b : 0) * p.ldl;
  if (valid && p.nparts > 0) {
    // split-K logits: the chunks' partial sums in split order, then the bias
    const float* pp = (const float*)((const char*)p.parts + wsoff) + (int64_t)b * p.ldp;
    const int64_t ps = (int64_t)B * p.ldp;
    for (int c = sub; c < C; c += CE_LANES) {
      float t = pp[c];
      for (int k = 1; k < p.nparts; ++k) t += pp[k * ps + c];
      zw[c] = t + p.bias[c];
    }
  }
  const float* z = zw;
  float mx = -INFINITY;
  if (valid)
    for (int c = sub; c < C; c += CE_LANES) mx = fmaxf(mx, z[c]);
#pragma unroll
  for (int off = 1; off < CE_LANES; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
  float s = 0.f;
  if (valid)
    for (int c = sub; c < C; c += CE_LANES) s += expf(z[c] - mx);
#pragma unroll
  for (int off = 1; off < CE_LANES; off <<= 1) s += __shfl_xor(s, off, 64);
  if (valid) {
    const int yb = y[b];
    if (sub == 0) rowloss[rl] = mx + logf(s) - z[yb];
    const float inv_s = 1.0f / s, invB = 1.0f / (float)B;
    for (int c = sub; c < C; c += CE_LANES) {
      const T g = TT<T>::from_f((expf(z[c] - mx) * inv_s - (c == yb ? 1.f : 0.f)) * invB);
      ((T*)p.G)[(int64_t)b * p.ldg + c] = g;
    }
  } else if (sub == 0) {
    rowloss[rl] = 0.f;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const int nrows = min(CE_ROWS, B - (int)blockIdx.x * CE_ROWS);
    float t = 0.f;
    for (int r = 0; r < nrows; ++r) t += rowloss[r];
    partial[(int64_t)p.model * pstride + blockIdx.x] = t;
  }
}

// One lane per problem of the list (the active models), writing that model's
// slot: its partials (row chunks, or the m-tiles of its fused logits GEMM)
// added in order.
__global__ void ce_finish_kernel(const CeProb* __restrict__ probs, const float* __restrict__ partial, int pstride,
                                 int nprobs, float* __restrict__ losses) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= nprobs) return;
  const int m = probs[i].model, n = probs[i].nchunks;
  float s = 0.f;
  for (int k = 0; k < n; ++k) s += partial[(int64_t)m * pstride + k];
  losses[m] = s * (1.0f / (float)probs[i].B);
}

// ---------------------------------------------------------------------------
// Self-attention core (AttnProb), one workgroup of 256 threads per (problem,
// sample). The sample's Q, K, V (and dA) rows are staged in LDS as fp32 with
// rows padded to d + 1 floats; every output element is one fmaf chain over
// its contraction index in ascending order, and the softmax row reductions
// are fixed lane-shuffle butterflies, so the result depends on nothing but
// the sample's own values.
// ---------------------------------------------------------------------------
template <typename T>
__device__ __forceinline__ void attn_stage(const AttnProb& p, int b, T* sQ, T* sK, T* sV) {
  // Q | K | V rows of 3d elements, copied as 16-byte vectors (d is a multiple
  // of 8) into LDS rows of d plus one 16-byte chunk, in the storage type
  constexpr int VEC = TT<T>::VEC;
  const int Tn = p.T, d = p.d, ld = d + VEC, vpr = d / VEC;
  const T* qkv = (const T*)p.QKV + (int64_t)b * Tn * p.ldq;
  for (int e = threadIdx.x; e < Tn * vpr; e += blockDim.x) {
    const int t = e / vpr, j = (e - t * vpr) * VEC;
    const T* row = qkv + (int64_t)t * p.ldq + j;
    *(u32x4*)(sQ + t * ld + j) = *(gptr<const u32x4>)row;
    *(u32x4*)(sK + t * ld + j) = *(gptr<const u32x4>)(row + d);
    *(u32x4*)(sV + t * ld + j) = *(gptr<const u32x4>)(row + 2 * d);
  }
}

// Four consecutive values of a row to global memory as one store (bf16: 8
// bytes, fp32: 16), or element by element at a row's end.
template <typename T>
__device__ __forceinline__ void attn_put4(T* dst, const float* v, int n, float scale) {
  if (n == 4) {
    if constexpr (sizeof(T) == 2) {
      u32x2 w;
      w[0] = f2bf2(v[0] * scale, v[1] * scale);
      w[1] = f2bf2(v[2] * scale, v[3] * scale);
      *(gptr<u32x2>)dst = w;
    } else {
      *(gptr<f32x4>)dst = f32x4{v[0] * scale, v[1] * scale, v[2] * scale, v[3] * scale};
    }
  } else {
    for (int e = 0; e < n; ++e) dst[e] = TT<T>::from_f(v[e] * scale);
  }
}

// out[r][c] = sum over x of a(r, x) * b(c, x) for r < rows, c < cols: each
// thread takes RB x CB blocks of outputs (columns fastest across threads), so
// one load of a(r, x) and of b(c, x) serves CB and RB multiply-adds. Every
// output is one fmaf chain over x in ascending order, as in the unblocked
// form; rows and columns past the end read a clamped valid element and are
// not stored. put(r, c0, v, n) receives the n valid values of row r from
// column c0.
template <int RB, int CB, class FA, class FB, class PUT>
__device__ __forceinline__ void attn_products(int rows, int cols, int n, FA&& fa, FB&& fb, PUT&& put) {
  const int nbc = (cols + CB - 1) / CB, nblk = ((rows + RB - 1) / RB) * nbc;
  for (int blk = threadIdx.x; blk < nblk; blk += blockDim.x) {
    const int r0 = (blk / nbc) * RB, c0 = (blk - (blk / nbc) * nbc) * CB;
    int rr[RB], cc[CB];
#pragma unroll
    for (int i = 0; i < RB; ++i) rr[i] = min(r0 + i, rows - 1);
#pragma unroll
    for (int j = 0; j < CB; ++j) cc[j] = min(c0 + j, cols - 1);
    float acc[RB][CB];
#pragma unroll
    for (int i = 0; i < RB; ++i)
#pragma unroll
      for (int j = 0; j < CB; ++j) acc[i][j] = 0.f;
    for (int x = 0; x < n; ++x) {
      float a[RB], b[CB];
#pragma unroll
      for (int i = 0; i < RB; ++i) a[i] = fa(rr[i], x);
#pragma unroll
      for (int j = 0; j < CB; ++j) b[j] = fb(cc[j], x);
#pragma unroll
      for (int i = 0; i < RB; ++i)
#pragma unroll
        for (int j = 0; j < CB; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    const int nc = min(CB, cols - c0);
#pragma unroll
    for (int i = 0; i < RB; ++i)
      if (r0 + i < rows) put(r0 + i, c0, acc[i], nc);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void attn_fwd_kernel(const AttnProb* __restrict__ probs,
                                                       const int32_t* __restrict__ tile_map) {
  extern __shared__ float sm[];
  const int pi = tile_map[2 * blockIdx.x], b = tile_map[2 * blockIdx.x + 1];
  if (pi < 0) return;
  const AttnProb& p = probs[pi];
  const int Tn = p.T, d = p.d, ld = d + TT<T>::VEC, ls = Tn + 1;
  T* sQ = (T*)sm;  // Q, K, V rows in the storage type, then [T][T + 1] fp32 scores
  T* sK = sQ + Tn * ld;
  T* sV = sK + Tn * ld;
  float* sS = (float*)(sV + Tn * ld);
  attn_stage<T>(p, b, sQ, sK, sV);
  __syncthreads();
  // S[i][t] = (Q K^T)[i][t] * scale
  attn_products<2, 2>(Tn, Tn, d, [&](int i, int k) { return TT<T>::to_f(sQ[i * ld + k]); },
                      [&](int t, int k) { return TT<T>::to_f(sK[t * ld + k]); },
                      [&](int i, int t0, const float* v, int n) {
                        for (int e = 0; e < n; ++e) sS[i * ls + t0 + e] = v[e] * p.scale;
                      });
  __syncthreads();
  // softmax over the keys: one wave per query row, lanes over the keys (T <= 64)
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  float* Pg = p.P + (int64_t)b * Tn * Tn;
  for (int i = wave; i < Tn; i += nw) {
    const float v = lane < Tn ? sS[i * ls + lane] : -INFINITY;
    const float mx = wave_max(v);
    const float ex = lane < Tn ? expf(v - mx) : 0.f;
    const float inv = 1.0f / wave_sum(ex);
    if (lane < Tn) {
      const float pr = ex * inv;
      sS[i * ls + lane] = pr;
      Pg[(int64_t)i * Tn + lane] = pr;
    }
  }
  __syncthreads();
  // A[i][j] = (P V)[i][j]
  T* A = (T*)p.A + (int64_t)b * Tn * p.lda;
  attn_products<4, 4>(Tn, d, Tn, [&](int i, int t) { return sS[i * ls + t]; },
                      [&](int j, int t) { return TT<T>::to_f(sV[t * ld + j]); },
                      [&](int i, int j0, const float* v, int n) { attn_put4<T>(A + (int64_t)i * p.lda + j0, v, n, 1.f); });
}

template <typename T>
__global__ __launch_bounds__(256) void attn_bwd_kernel(const AttnProb* __restrict__ probs,
                                                       const int32_t* __restrict__ tile_map) {
  extern __shared__ float sm[];
  const int pi = tile_map[2 * blockIdx.x], b = tile_map[2 * blockIdx.x + 1];
  if (pi < 0) return;
  const AttnProb& p = probs[pi];
  constexpr int VEC = TT<T>::VEC;
  const int Tn = p.T, d = p.d, ld = d + VEC, ls = Tn + 1;
  T* sQ = (T*)sm;  // Q, K, V, dA rows in the storage type, then two fp32 tiles
  T* sK = sQ + Tn * ld;
  T* sV = sK + Tn * ld;
  T* sD = sV + Tn * ld;                       // dA
  float* sP = (float*)(sD + Tn * ld);         // [T][T + 1] probabilities
  float* sG = sP + Tn * ls;                   // [T][T + 1] dP, then dS
  attn_stage<T>(p, b, sQ, sK, sV);
  const T* dA = (const T*)p.dA + (int64_t)b * Tn * p.lda;
  const float* Pg = p.P + (int64_t)b * Tn * Tn;
  {
    const int vpr = d / VEC;
    for (int e = threadIdx.x; e < Tn * vpr; e += blockDim.x) {
      const int i = e / vpr, j = (e - i * vpr) * VEC;
      *(u32x4*)(sD + i * ld + j) = *(gptr<const u32x4>)(dA + (int64_t)i * p.lda + j);
    }
  }
  for (int e = threadIdx.x; e < Tn * Tn; e += blockDim.x) {
    const int i = e / Tn, t = e - i * Tn;
    sP[i * ls + t] = Pg[e];
  }
  __syncthreads();
  // dP[i][t] = sum_j dA[i][j] V[t][j]
  attn_products<2, 2>(Tn, Tn, d, [&](int i, int j) { return TT<T>::to_f(sD[i * ld + j]); },
                      [&](int t, int j) { return TT<T>::to_f(sV[t * ld + j]); },
                      [&](int i, int t0, const float* v, int n) {
                        for (int e = 0; e < n; ++e) sG[i * ls + t0 + e] = v[e];
                      });
  __syncthreads();
  // dS = P * (dP - rowsum(P * dP)), one wave per row
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  for (int i = wave; i < Tn; i += nw) {
    const float pr = lane < Tn ? sP[i * ls + lane] : 0.f;
    const float dp = lane < Tn ? sG[i * ls + lane] : 0.f;
    const float rd = wave_sum(pr * dp);
    if (lane < Tn) sG[i * ls + lane] = pr * (dp - rd);
  }
  __syncthreads();
  T* dqkv = (T*)p.dQKV + (int64_t)b * Tn * p.ldq;
  // dQ[r][k] = scale * sum_t dS[r][t] K[t][k]
  attn_products<4, 4>(Tn, d, Tn, [&](int r, int t) { return sG[r * ls + t]; },
                      [&](int k, int t) { return TT<T>::to_f(sK[t * ld + k]); },
                      [&](int r, int k0, const float* v, int n) { attn_put4<T>(dqkv + (int64_t)r * p.ldq + k0, v, n, p.scale); });
  // dK[r][k] = scale * sum_i dS[i][r] Q[i][k]
  attn_products<4, 4>(Tn, d, Tn, [&](int r, int i) { return sG[i * ls + r]; },
                      [&](int k, int i) { return TT<T>::to_f(sQ[i * ld + k]); },
                      [&](int r, int k0, const float* v, int n) {
                        attn_put4<T>(dqkv + (int64_t)r * p.ldq + d + k0, v, n, p.scale);
                      });
  // dV[r][k] = sum_i P[i][r] dA[i][k]
  attn_products<4, 4>(Tn, d, Tn, [&](int r, int i) { return sP[i * ls + r]; },
                      [&](int k, int i) { return TT<T>::to_f(sD[i * ld + k]); },
                      [&](int r, int k0, const float* v, int n) {
                        attn_put4<T>(dqkv + (int64_t)r * p.ldq + 2 * d + k0, v, n, 1.f);
                      });
}

// ---------------------------------------------------------------------------
// Multi-tensor SGD (64x64 tiles; the transposed copy goes through LDS).
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void sgd_kernel(const SgdTensor* __restrict__ ts,
                                                  const int32_t* __restrict__ tile_tensor, int blk0, float lr,
                                                  int use_grad) {
  __shared__ float sm[SGD_TILE][SGD_TILE + 1];
  const int blk = blockIdx.x + blk0;  // the launch covers tiles [blk0, blk0 + gridDim.x) of the table
  const SgdTensor& t = ts[tile_tensor[blk]];
  const int local = blk - t.tile_base;
  const int per_tap = t.tiles_r * t.tiles_c;
  const int j = local / per_tap, rem = local - j * per_tap;
  const int tr = rem / t.tiles_c, tc = rem - tr * t.tiles_c;
  const int r0 = tr * SGD_TILE, c0 = tc * SGD_TILE;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const int rl = ty + 16 * s, r = r0 + rl;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int cl = 4 * tx + e, c = c0 + cl;
      if (r < t.R && c < t.Cc) {
        const int64_t idx = (int64_t)r * t.ldw + (int64_t)j * t.Cc + c;
        float w = t.W[idx];
        if (use_grad) {
          w = fmaf(-lr, t.G[idx], w);
          t.W[idx] = w;
        }
        if (t.Wb) ((bf16_t*)t.Wb)[idx] = f2bf(w);
        sm[rl][cl] = w;
      }
    }
  }
  if (!t.WT) return;
  __syncthreads();
  // WT[c][j*R + r]: consecutive threads take consecutive r for coalescing
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const int cl = ty + 16 * s, c = c0 + cl;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int rl = 4 * tx + e, r = r0 + rl;
      if (r < t.R && c < t.Cc) store_t<T>(t.WT, (int64_t)c * t.ldwt + (int64_t)j * t.R + r, sm[rl][cl]);
    }
  }
}

// ---------------------------------------------------------------------------
// Batch load: fp32 NCHW -> storage-type NHWC (+ NHWC with Cs stored channels).
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void load_kernel(const float* __restrict__ x, int B, int C, int H, int W,
                                                   T* __restrict__ X, T* __restrict__ XC, int Cs) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t total = (int64_t)B * C * H * W;
  if (e >= total) return;
  const int hw = H * W;
  const int64_t b = e / ((int64_t)C * hw);
  const int rem = (int)(e - b * C * hw);
  const int c = rem / hw, s = rem - c * hw;
  const T v = TT<T>::from_f(x[e]);
  if (X) X[(b * hw + s) * C + c] = v;
  if (XC) XC[(b * hw + s) * Cs + c] = v;
}

// ---------------------------------------------------------------------------
// Launch wrappers
// ---------------------------------------------------------------------------
hipError_t launch_gemm(bool bf16, bool bwd, const GemmProb* probs, const int32_t* tile_map, int ntiles, float lr,
                       const float* lrv, const OptHp* opt, bool keep_grads, const int32_t* labels,
                       bool per_model_labels, int64_t wsoff, hipStream_t s) {
  if (ntiles <= 0) return hipSuccess;
  auto go = [&](auto kern, int nt) {
    hipLaunchKernelGGL(kern, dim3(ntiles), dim3(nt), 0, s, probs, tile_map, lr, lrv, opt, (int)keep_grads, labels,
                       (int)per_model_labels, wsoff);
  };
  if (bf16) {
    constexpr int NT = GemmMma<bf16_t, GEMM_BM_BF16, GEMM_BN_BF16, GEMM_BK_BF16>::NT;
    if (!bwd) go(gemm_kernel<bf16_t, GEMM_BM_BF16, GEMM_BN_BF16, GEMM_BK_BF16, false, false>, NT);
    else if (opt) go(gemm_kernel<bf16_t, GEMM_BM_BF16, GEMM_BN_BF16, GEMM_BK_BF16, true, true>, NT);
    else go(gemm_kernel<bf16_t, GEMM_BM_BF16, GEMM_BN_BF16, GEMM_BK_BF16, false, true>, NT);
  } else {
    if (!bwd) go(gemm_kernel<float, GEMM_BM_F32, GEMM_BN_F32, GEMM_BK_F32, false, false>, 256);
    else if (opt) go(gemm_kernel<float, GEMM_BM_F32, GEMM_BN_F32, GEMM_BK_F32, true, true>, 256);
    else go(gemm_kernel<float, GEMM_BM_F32, GEMM_BN_F32, GEMM_BK_F32, false, true>, 256);
  }
  return hipGetLastError();
}

hipError_t launch_conv_fwd(bool bf16, const ConvProb* probs, const int32_t* tile_map, int ntiles, hipStream_t s) {
  if (ntiles <= 0) return hipSuccess;
  if (bf16)
    hipLaunchKernelGGL((conv_fwd_kernel<bf16_t, CONV_BM_BF16, CONV_BN_BF16, CONV_BK_BF16>), dim3(ntiles), dim3(256),
                       0, s, probs, tile_map);
  else
    hipLaunchKernelGGL((conv_fwd_kernel<float, CONV_BM_F32, CONV_BN_F32, CONV_BK_F32>), dim3(ntiles), dim3(256), 0,
                       s, probs, tile_map);
  return hipGetLastError();
}

hipError_t launch_conv_dgrad(bool bf16, const ConvProb* probs, const int32_t* tile_map, int ntiles, hipStream_t s) {
  if (ntiles <= 0) return hipSuccess;
  if (bf16)
    hipLaunchKernelGGL((conv_dgrad_kernel<bf16_t, CONV_BM_BF16, CONV_BN_BF16, CONV_BK_BF16>), dim3(ntiles),
                       dim3(256), 0, s, probs, tile_map);
  else
    hipLaunchKernelGGL((conv_dgrad_kernel<float, CONV_BM_F32, CONV_BN_F32, CONV_BK_F32>), dim3(ntiles), dim3(256),
                       0, s, probs, tile_map);
  return hipGetLastError();
}

hipError_t launch_conv_halo(bool bf16, bool dgrad, const ConvProb* probs, const int32_t* tile_map, int ntiles,
                            size_t lds_bytes, hipStream_t s) {
  if (ntiles <= 0) return hipSuccess;
  // allow dynamic LDS up to the halo budget (above the default cap)
  static const hipError_t attr = [] {
    hipError_t e = hipSuccess, r;
    r = hipFuncSetAttribute(reinterpret_cast<const void*>(&conv_halo_kernel<bf16_t, CONV_BM_BF16, CONV_BN_BF16, CONV_BK_BF16, true>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, HALO_LDS_BF16);
    if (r != hipSuccess) e = r;
    r = hipFuncSetAttribute(reinterpret_cast<const void*>(&conv_halo_kernel<bf16_t, CONV_BM_BF16, CONV_BN_BF16, CONV_BK_BF16, false>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, HALO_LDS_BF16);
    if (r != hipSuccess) e = r;
    r = hipFuncSetAttribute(reinterpret_cast<const void*>(&conv_halo_kernel<float, CONV_BM_F32, CONV_BN_F32, CONV_BK_F32, true>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, HALO_LDS_F32);
    if (r != hipSuccess) e = r;
    r = hipFuncSetAttribute(reinterpret_cast<const void*>(&conv_halo_kernel<float, CONV_BM_F32, CONV_BN_F32, CONV_BK_F32, false>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, HALO_LDS_F32);
    if (r != hipSuccess) e = r;
    return e;
  }();
  if (attr != hipSuccess) return attr;
  if (bf16) {
    constexpr int NT = 64 * halo_waves<bf16_t>();
    if (dgrad)
      hipLaunchKernelGGL((conv_halo_kernel<bf16_t, CONV_BM_BF16, CONV_BN_BF16, CONV_BK_BF16, true>), dim3(ntiles),
                         dim3(NT), lds_bytes, s, probs, tile_map);
    else
      hipLaunchKernelGGL((conv_halo_kernel<bf16_t, CONV_BM_BF16, CONV_BN_BF16, CONV_BK_BF16, false>), dim3(ntiles),
                         dim3(NT), lds_bytes, s, probs, tile_map);
  } else {
    if (dgrad)
      hipLaunchKernelGGL((conv_halo_kernel<float, CONV_BM_F32, CONV_BN_F32, CONV_BK_F32, true>), dim3(ntiles),
                         dim3(256), lds_bytes, s, probs, tile_map);
    else
      hipLaunchKernelGGL((conv_halo_kernel<float, CONV_BM_F32, CONV_BN_F32, CONV_BK_F32, false>), dim3(ntiles),
                         dim3(256), lds_bytes, s, probs, tile_map);
  }
  return hipGetLastError();
}

hipError_t launch_conv_wgrad(bool bf16, int mode, const ConvProb* probs, const int32_t* tile_map, int ntiles,
                             int64_t wsoff, hipStream_t s) {
  if (ntiles <= 0) return hipSuccess;
#define UN_WGRAD_LAUNCH(T, BM, BN, BK, M) \
  hipLaunchKernelGGL((conv_wgrad_kernel<T, BM, BN, BK, M>), dim3(ntiles), dim3(256), 0, s, probs, tile_map, wsoff)
  if (bf16) {
    constexpr int NT = GemmMma<bf16_t, CONV_BM_BF16, CONV_BN_BF16, CONV_BK_BF16, 4, 4>::NT;
    const bool narrow = (mode & WG_NARROW) != 0;
    mode &= ~WG_NARROW;
    if (mode == WG_POOLED && narrow)
      hipLaunchKernelGGL((conv_wgrad_mfma_kernel<true, true>), dim3(ntiles), dim3(NT / 2), 0, s, probs, tile_map, wsoff);
    else if (mode == WG_POOLED)
      hipLaunchKernelGGL((conv_wgrad_mfma_kernel<true, false>), dim3(ntiles), dim3(NT), 0, s, probs, tile_map, wsoff);
    else if (mode == WG_PLAIN && narrow)
      hipLaunchKernelGGL((conv_wgrad_mfma_kernel<false, true>), dim3(ntiles), dim3(NT / 2), 0, s, probs, tile_map, wsoff);
    else if (mode == WG_PLAIN)
      hipLaunchKernelGGL((conv_wgrad_mfma_kernel<false, false>), dim3(ntiles), dim3(NT), 0, s, probs, tile_map, wsoff);
    else UN_WGRAD_LAUNCH(bf16_t, CONV_BM_BF16, CONV_BN_BF16, CONV_BK_BF16, WG_GENERIC);
  } else {
    if (mode == WG_POOLED) UN_WGRAD_LAUNCH(float, CONV_BM_F32, CONV_BN_F32, CONV_BK_F32, WG_POOLED);
    else if (mode == WG_PLAIN) UN_WGRAD_LAUNCH(float, CONV_BM_F32, CONV_BN_F32, CONV_BK_F32, WG_PLAIN);
    else UN_WGRAD_LAUNCH(float, CONV_BM_F32, CONV_BN_F32, CONV_BK_F32, WG_GENERIC);
  }
#undef UN_WGRAD_LAUNCH
  return hipGetLastError();
}

hipError_t launch_reduce(bool bf16, const ReduceProb* probs, const int32_t* blk_prob, int nblocks, float lr,
                         const float* lrv, const OptHp* opt, bool keep_grads, int64_t wsoff, hipStream_t s) {
  if (nblocks <= 0) return hipSuccess;
  if (bf16)
    hipLaunchKernelGGL(reduce_kernel<bf16_t>, dim3(nblocks), dim3(REDUCE_BLOCK), 0, s, probs, blk_prob, lr, lrv, opt,
                       (int)keep_grads, wsoff);
  else
    hipLaunchKernelGGL(reduce_kernel<float>, dim3(nblocks), dim3(REDUCE_BLOCK), 0, s, probs, blk_prob, lr, lrv, opt,
                       (int)keep_grads, wsoff);
  return hipGetLastError();
}

// Values passed by value in the kernel arguments, SETV_CHUNK per launch: no
// host buffer has to outlive the call.
constexpr int SETV_CHUNK = 256;
struct SetValues {
  float v[SETV_CHUNK];
};
__global__ void set_values_kernel(float* __restrict__ dst, SetValues vals, int n) {
  const int i = threadIdx.x;
  if (i < n) dst[i] = vals.v[i];
}

hipError_t launch_set_values(float* dst, const float* vals, int n, hipStream_t s) {
  for (int i0 = 0; i0 < n; i0 += SETV_CHUNK) {
    const int k = n - i0 < SETV_CHUNK ? n - i0 : SETV_CHUNK;
    SetValues sv{};
    for (int i = 0; i < k; ++i) sv.v[i] = vals[i0 + i];
    hipLaunchKernelGGL(set_values_kernel, dim3(1), dim3(SETV_CHUNK), 0, s, dst + i0, sv, k);
  }
  return hipGetLastError();
}

hipError_t launch_attn(bool bf16, bool bwd, const AttnProb* probs, const int32_t* tile_map, int nblocks,
                       size_t lds_bytes, hipStream_t s) {
  if (nblocks <= 0) return hipSuccess;
  if (lds_bytes > (size_t)160 * 1024) return hipErrorInvalidValue;
  // allow dynamic LDS up to the whole 160 KiB of a CU (above the default cap)
  static const hipError_t attr = [] {
    hipError_t e = hipSuccess, r;
    const void* k[4] = {reinterpret_cast<const void*>(&attn_fwd_kernel<bf16_t>),
                        reinterpret_cast<const void*>(&attn_fwd_kernel<float>),
                        reinterpret_cast<const void*>(&attn_bwd_kernel<bf16_t>),
                        reinterpret_cast<const void*>(&attn_bwd_kernel<float>)};
    for (const void* f : k) {
      r = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
      if (r != hipSuccess) e = r;
    }
    return e;
  }();
  if (attr != hipSuccess) return attr;
  if (bwd) {
    if (bf16)
      hipLaunchKernelGGL(attn_bwd_kernel<bf16_t>, dim3(nblocks), dim3(256), lds_bytes, s, probs, tile_map);
    else
      hipLaunchKernelGGL(attn_bwd_kernel<float>, dim3(nblocks), dim3(256), lds_bytes, s, probs, tile_map);
  } else {
    if (bf16)
      hipLaunchKernelGGL(attn_fwd_kernel<bf16_t>, dim3(nblocks), dim3(256), lds_bytes, s, probs, tile_map);
    else
      hipLaunchKernelGGL(attn_fwd_kernel<float>, dim3(nblocks), dim3(256), lds_bytes, s, probs, tile_map);
  }
  return hipGetLastError();
}

hipError_t launch_ce(bool bf16, const CeProb* probs, int nprobs, int nrows, const int32_t* labels,
                     bool per_model_labels, int maxB, float* partial, int pstride, float* losses, int64_t wsoff,
                     hipStream_t s) {
  if (nprobs <= 0) return hipSuccess;
  const int nchunks = (maxB + CE_ROWS - 1) / CE_ROWS;
  if (nrows > 0) {
    if (bf16)
      hipLaunchKernelGGL(ce_rows_kernel<bf16_t>, dim3(nchunks, nrows), dim3(CE_ROWS * CE_LANES), 0, s, probs, labels,
                         (int)per_model_labels, partial, pstride, wsoff);
    else
      hipLaunchKernelGGL(ce_rows_kernel<float>, dim3(nchunks, nrows), dim3(CE_ROWS * CE_LANES), 0, s, probs, labels,
                         (int)per_model_labels, partial, pstride, wsoff);
  }
  hipLaunchKernelGGL(ce_finish_kernel, dim3((nprobs + 63) / 64), dim3(64), 0, s, probs, partial, pstride, nprobs,
                     losses);
  return hipGetLastError();
}

hipError_t launch_sgd(bool bf16, const SgdTensor* t, const int32_t* tile_tensor, int blk0, int ntiles, float lr,
                      bool use_grad, hipStream_t s) {
  if (ntiles <= 0) return hipSuccess;
  if (bf16)
    hipLaunchKernelGGL(sgd_kernel<bf16_t>, dim3(ntiles), dim3(256), 0, s, t, tile_tensor, blk0, lr, (int)use_grad);
  else
    hipLaunchKernelGGL(sgd_kernel<float>, dim3(ntiles), dim3(256), 0, s, t, tile_tensor, blk0, lr, (int)use_grad);
  return hipGetLastError();
}

hipError_t launch_load(bool bf16, const float* x, int B, int C, int H, int W, void* X,
                       void* XC, int Cs, hipStream_t s) {
  const int64_t total = (int64_t)B * C * H * W;
  const int blocks = (int)((total + 255) / 256);
  if (blocks <= 0) return hipSuccess;
  if (bf16)
    hipLaunchKernelGGL(load_kernel<bf16_t>, dim3(blocks), dim3(256), 0, s, x, B, C, H, W, (bf16_t*)X, (bf16_t*)XC,
                       Cs);
  else
    hipLaunchKernelGGL(load_kernel<float>, dim3(blocks), dim3(256), 0, s, x, B, C, H, W, (float*)X, (float*)XC, Cs);
  return hipGetLastError();
}

}  // namespace un
