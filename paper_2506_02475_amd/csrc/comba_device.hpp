// Device building blocks for the gfx950 (CDNA4) Comba kernels.
//
// Every dense contraction in the chunk-wise algorithm is a product of 16x16
// output tiles computed by one 64-lane wavefront with MFMA.  Operands are staged
// in LDS with the reduction (k) index contiguous, so a lane fetches its 8 (bf16
// MFMA) k-values with one or two vector LDS reads.
//
// Precision policy.  bf16 inputs (q, k, v, beta, dO) are exact in bf16.  Every
// other operand (the inverse M, the masked gate/score matrices, states, pseudo
// values and their gradients) is fp32; when it meets a bf16 MFMA it is split
// into hi = bf16(x) and lo = bf16(x - hi), and the product keeps the hi*hi,
// hi*lo and lo*hi terms (about 16 significant bits per fp32 operand, fp32
// accumulation).  With fp32 inputs the fp32 MFMA (16x16x4) is used throughout.
//
// MFMA register layouts used below (wave64, 16x16 tiles):
//   A operand (16 x K): lane l supplies row (l % 16), k-group (l / 16)
//   B operand (K x 16): lane l supplies column (l % 16), k-group (l / 16)
//   accumulator:        lane l holds column (l % 16), rows 4*(l/16) + i, i = 0..3
// The order of k inside a group only has to agree between A and B.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace comba {

constexpr int CH = 64;        // chunk length (tokens)
constexpr int NTHR = 256;     // threads per workgroup: 4 wavefronts
constexpr int NWAVE = 4;

typedef uint16_t bf16_t;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

template <typename T> struct is_f32 { static constexpr bool value = false; };
template <> struct is_f32<float> { static constexpr bool value = true; };

__device__ __forceinline__ float bf2f(bf16_t b) { return __uint_as_float(((uint32_t)b) << 16); }
__device__ __forceinline__ float to_f(float x) { return x; }
__device__ __forceinline__ float to_f(bf16_t x) { return bf2f(x); }

// Storage padding (elements) that keeps 16-byte row alignment and spreads the
// 16 rows read by one MFMA operand fetch over distinct LDS banks.
template <typename T> struct Pad { static constexpr int value = 16 / sizeof(T); };

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }
__device__ __forceinline__ int wave_id() { return threadIdx.x >> 6; }
// The same in a scalar register: the compiler cannot tell on its own that it is
// uniform across the wave, and a per-lane copy makes every branch and address
// derived from it per-lane.  (For the streaming prologue kernels, whose loop
// control derives from it; in the scan kernels the scalar form changed the
// schedule for the worse: the d = 256 forward scan took 12% longer.)
__device__ __forceinline__ int wave_id_s() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

__device__ __forceinline__ floatx4 zero4() { return floatx4{0.f, 0.f, 0.f, 0.f}; }

// IEEE 754-2019 maximum: a NaN operand gives NaN (fmaxf would drop it).  The
// block maxima behind every int16 scale use it, so that a non-finite value
// turns its block's scale into NaN (see q_scale) instead of vanishing.  On
// gfx950 it is v_maximum3_f32, which also folds |x| and a third operand.
__device__ __forceinline__ float nmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }
__device__ __forceinline__ float nmax_abs4(float m, const floatx4& x) {
  return nmax(nmax(m, nmax(fabsf(x[0]), fabsf(x[1]))), nmax(fabsf(x[2]), fabsf(x[3])));
}

template <int MT, int NT>
__device__ __forceinline__ void zero_acc(floatx4 (&acc)[MT][NT]) {
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[i][j] = zero4();
}

// ---- operand fragments -------------------------------------------------------

// 8 consecutive-k bf16 values of an exact operand.
__device__ __forceinline__ bf16x8 frag_exact(const bf16_t* p) {
  return *reinterpret_cast<const bf16x8*>(p);
}

// 8 consecutive-k fp32 values split into bf16 hi and lo parts.
__device__ __forceinline__ void frag_split(const float* p, bf16x8& hi, bf16x8& lo) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  const float4 b = *reinterpret_cast<const float4*>(p + 4);
  const float x[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const __bf16 h = (__bf16)x[e];
    hi[e] = h;
    lo[e] = (__bf16)(x[e] - (float)h);
  }
}

template <typename T> struct Frag;
template <> struct Frag<bf16_t> {
  bf16x8 hi;
  __device__ __forceinline__ void load(const bf16_t* p) { hi = frag_exact(p); }
  static constexpr bool split = false;
};
template <> struct Frag<float> {
  bf16x8 hi, lo;
  __device__ __forceinline__ void load(const float* p) { frag_split(p, hi, lo); }
  static constexpr bool split = true;
};

// acc[mt][nt] += sum_{k < K} A(16 mt + i, k) * B(k, 16 nt + j)
//   A(m, k) = A[m * lda + k]   (row-major, k contiguous)
//   B(k, n) = B[n * ldb + k]   (stored transposed, k contiguous)
// F32 selects the fp32 MFMA (both operands fp32); otherwise the bf16 MFMA with
// fp32 operands split as described above.
template <bool F32, int MT, int NT, int K, typename TA, typename TB>
__device__ __forceinline__ void mma(floatx4 (&acc)[MT][NT], const TA* __restrict__ A, int lda,
                                    const TB* __restrict__ B, int ldb) {
  const int lane = lane_id();
  const int r = lane & 15, grp = lane >> 4;
  if constexpr (F32) {
    static_assert(is_f32<TA>::value && is_f32<TB>::value, "fp32 MFMA takes fp32 operands");
#pragma unroll
    for (int k0 = 0; k0 < K; k0 += 4) {
      float a[MT], b[NT];
#pragma unroll
      for (int i = 0; i < MT; ++i) a[i] = A[(16 * i + r) * lda + k0 + grp];
#pragma unroll
      for (int j = 0; j < NT; ++j) b[j] = B[(16 * j + r) * ldb + k0 + grp];
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  } else {
    static_assert(K % 32 == 0, "bf16 MFMA reduces 32 at a time");
#pragma unroll
    for (int k0 = 0; k0 < K; k0 += 32) {
      const int kk = k0 + 8 * grp;
      Frag<TA> a[MT];
      Frag<TB> b[NT];
#pragma unroll
      for (int i = 0; i < MT; ++i) a[i].load(A + (16 * i + r) * lda + kk);
#pragma unroll
      for (int j = 0; j < NT; ++j) b[j].load(B + (16 * j + r) * ldb + kk);
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j) {
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i].hi, b[j].hi, acc[i][j], 0, 0, 0);
          if constexpr (Frag<TA>::split)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i].lo, b[j].hi, acc[i][j], 0, 0, 0);
          if constexpr (Frag<TB>::split)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i].hi, b[j].lo, acc[i][j], 0, 0, 0);
        }
    }
  }
}

// Row / column of accumulator element e of tile (mt, nt), relative to the
// block origin passed to mma().
__device__ __forceinline__ int acc_row(int mt, int e) { return 16 * mt + 4 * (lane_id() >> 4) + e; }
__device__ __forceinline__ int acc_col(int nt) { return 16 * nt + (lane_id() & 15); }

// ---- accumulator row stores --------------------------------------------------
// An accumulator tile gives lane l the rows 4 (l / 16) + e (e = 0..3) of
// column l % 16, so a plain store writes 4 bytes per lane.  quad_transpose
// exchanges values inside each group of four lanes (DPP quad permutations, no
// LDS) so that lane l instead holds row 4 (l / 16) + (l % 4), columns
// (l & 12) + e: four consecutive columns of one row, written with one 16-byte
// store.  Two butterfly rounds: exchange with lane ^ 1, then with lane ^ 2.
template <int CTRL>
__device__ __forceinline__ float dpp_quad(float x) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), CTRL, 0xF, 0xF, true));
}
__device__ __forceinline__ floatx4 quad_transpose(floatx4 a) {
  constexpr int XOR1 = 0xB1;  // quad_perm [1, 0, 3, 2]
  constexpr int XOR2 = 0x4E;  // quad_perm [2, 3, 0, 1]
  const int i = lane_id() & 3;
  const bool odd = i & 1, hi = i & 2;
  {
    const float r0 = dpp_quad<XOR1>(odd ? a[0] : a[1]);
    const float r1 = dpp_quad<XOR1>(odd ? a[2] : a[3]);
    a[0] = odd ? r0 : a[0];
    a[1] = odd ? a[1] : r0;
    a[2] = odd ? r1 : a[2];
    a[3] = odd ? a[3] : r1;
  }
  {
    const float r0 = dpp_quad<XOR2>(hi ? a[0] : a[2]);
    const float r1 = dpp_quad<XOR2>(hi ? a[1] : a[3]);
    a[0] = hi ? r0 : a[0];
    a[2] = hi ? a[2] : r0;
    a[1] = hi ? r1 : a[1];
    a[3] = hi ? a[3] : r1;
  }
  return a;
}
// Row and first column (relative to the tile origin) of the four values a lane
// holds after quad_transpose.
__device__ __forceinline__ int qt_row() { return 4 * (lane_id() >> 4) + (lane_id() & 3); }
__device__ __forceinline__ int qt_col() { return lane_id() & 12; }
__device__ __forceinline__ void store4(float* p, const floatx4& x) {
  *reinterpret_cast<float4*>(p) = make_float4(x[0], x[1], x[2], x[3]);
}
// An element at a per-lane byte offset from a wave-uniform base pointer: the
// compiler keeps the base in SGPRs and the offset in one VGPR (global
// addressing with a scalar base), instead of 64-bit per-lane address arithmetic.
// The offset is unsigned 32-bit: callers keep it below 2^32 (offsets inside one
// chunk or chunk-head).
template <typename T>
__device__ __forceinline__ T& at(T* base, unsigned byte_off) {
  return *reinterpret_cast<T*>(reinterpret_cast<char*>(base) + byte_off);
}
template <typename T>
__device__ __forceinline__ const T& at(const T* base, unsigned byte_off) {
  return *reinterpret_cast<const T*>(reinterpret_cast<const char*>(base) + byte_off);
}
// Stores through a raw buffer whose record count ends at byte nbytes of g: the
// hardware drops every store at or past it, so the rows past a chunk end need
// no branch around their stores (g 4-byte aligned).  The record count is an
// unsigned 32-bit field: a chunk's rows at H <= 65535 heads of up to 256
// values span less than 2^32 bytes.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t clip_rsrc(float* g, unsigned nbytes) {
  return __builtin_amdgcn_make_buffer_rsrc(g, 0, (int)nbytes, 0x00020000);
}
__device__ __forceinline__ void store_clip(float x, __amdgpu_buffer_rsrc_t rs, unsigned byte_off) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(x), rs, byte_off, 0, 0);
}
__device__ __forceinline__ void store_clip4(const floatx4& x, __amdgpu_buffer_rsrc_t rs, unsigned byte_off) {
  typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
  const u32x4_t u = {__float_as_uint(x[0]), __float_as_uint(x[1]), __float_as_uint(x[2]), __float_as_uint(x[3])};
  __builtin_amdgcn_raw_buffer_store_b128(u, rs, byte_off, 0, 0);
}

// Max over the four lanes r16, r16 + 16, r16 + 32, r16 + 48 (the lanes that
// hold one row of a transposed MFMA accumulator) of values >= 0 or NaN:
// v_permlane16_swap / v_permlane32_swap with both operands x hand lane l the
// values of lanes l & ~16 and l | 16 (resp. 32) (checked with an in-bounds
// probe); non-negative floats order like their bit patterns, and every NaN
// pattern lies above +Inf, so a NaN wins.
__device__ __forceinline__ float rowgroup_max(float m) {
  const unsigned x = __float_as_uint(m);
  const auto a = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  const unsigned y = max(a[0], a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(y, y, false, false);
  return __uint_as_float(max(b[0], b[1]));
}

// ---- int16 fixed-point row blocks -----------------------------------------
// The chunk states and pseudo-values that the scans hand to the backward
// gradient kernel are stored as int16 q with one power-of-two scale s per
// (row, 32-column block): x = q * s, s = 2^(e - 15) where the block's max |x| is
// below 2^e, so |q| <= 32767 and the rounding error is at most s / 2, i.e. at
// most 2^-15 of the block's max.  q * s splits exactly into the bf16 (hi, lo)
// pair the consumer's MFMA products use, so no further rounding is added there.
// Zero and tiny maxima give a scale in [2^-115, 2^113].  A block whose max is
// Inf or NaN (a non-finite value in the block, found by the NaN-propagating
// maxima) gets the scale NaN: every value decoded from it is NaN, so
// non-finite inputs stay visible downstream instead of saturating to +-32767.
__device__ __forceinline__ int q_exponent(float m) {  // e with m < 2^e, m >= 0
  return max(((__float_as_int(m) >> 23) & 0xFF) - 126, -100);
}
__device__ __forceinline__ float q_scale(float m) {
  const int e = q_exponent(m);  // 129: exponent field 255, m is Inf or NaN
  return e > 128 ? __int_as_float(0x7FC00000) : __int_as_float((e + 112) << 23);
}
// 1 / s, divided by 32767 for the snorm16 conversion in q_pack4
__device__ __forceinline__ float q_inv_scale(float m) {
  return __int_as_float((142 - q_exponent(m)) << 23) * (1.0f / 32767.0f);
}
// four values (times the inverse scale) -> four int16 q = round(x / s),
// saturated to +-32767: v_cvt_pknorm_i16_f32 rounds 32767 y to the nearest
// integer after clamping y to [-1, 1] and packs two results (first argument in
// the low half; checked on the device with an in-bounds probe).  The factor
// 1/32767 in the inverse scale is rounded, so q can differ from round(x / s)
// by one only where x / s lies within 2^-9 of a half-integer.
__device__ __forceinline__ uint2 q_pack4(const floatx4& x, float inv) {
  const auto a = __builtin_amdgcn_cvt_pknorm_i16(x[0] * inv, x[1] * inv);
  const auto b = __builtin_amdgcn_cvt_pknorm_i16(x[2] * inv, x[3] * inv);
  return make_uint2(__builtin_bit_cast(uint32_t, a), __builtin_bit_cast(uint32_t, b));
}
// The same with one inverse scale per value (four columns with column scales).
__device__ __forceinline__ uint2 q_pack4v(const floatx4& x, const floatx4& inv) {
  const auto a = __builtin_amdgcn_cvt_pknorm_i16(x[0] * inv[0], x[1] * inv[1]);
  const auto b = __builtin_amdgcn_cvt_pknorm_i16(x[2] * inv[2], x[3] * inv[3]);
  return make_uint2(__builtin_bit_cast(uint32_t, a), __builtin_bit_cast(uint32_t, b));
}
__device__ __forceinline__ float4 q_unpack4(uint2 u, float s) {
  return make_float4((float)(int)(int16_t)(u.x & 0xFFFFu) * s, (float)((int)u.x >> 16) * s,
                     (float)(int)(int16_t)(u.y & 0xFFFFu) * s, (float)((int)u.y >> 16) * s);
}

// Wider stores of a 32-column int16 row block: a lane (group g = lane / 16)
// holds the 4-column pieces a (columns 4g .. 4g+3) and b (16 + 4g ..) of its
// row.  One v_permlane16_swap per dword exchanges b of the even groups with a
// of the odd ones, after which groups 0, 1, 2, 3 hold the 8 consecutive
// columns 0-7, 16-23, 8-15, 24-31 (checked with an in-bounds probe): one
// 16-byte store per lane and row instead of two 8-byte ones.  (Each store
// instruction costs the scans' single wave per SIMD about as much as the
// arithmetic that produced it, whatever its width.)
__device__ __forceinline__ uint4 row8_from_pieces(uint2 a, uint2 b) {
  const auto x = __builtin_amdgcn_permlane16_swap(a.x, b.x, false, false);
  const auto y = __builtin_amdgcn_permlane16_swap(a.y, b.y, false, false);
  return make_uint4(x[0], y[0], x[1], y[1]);
}
// First column of the 8 a lane holds after row8_from_pieces.
__device__ __forceinline__ int row8_col() {
  const int g = lane_id() >> 4;
  return 8 * (((g & 1) << 1) | (g >> 1));
}

// Two fp32 values as packed bf16 (hi, lo): hi = bf16(x) (nearest), lo =
// bf16(x - hi), each pair converted by one v_cvt_pk_bf16_f32 (3 VALU per value).
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void split2(float a, float b, uint32_t& hi, uint32_t& lo) {
  const uint32_t h = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
  const float ah = __uint_as_float(h << 16), bh = __uint_as_float(h & 0xFFFF0000u);
  hi = h;
  lo = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a - ah, b - bh}, bf16x2_t));
}

// Eight int16 (one 16-byte piece of a stored row) as the exact bf16 pair
// hi + lo of each value: |q| < 2^15, hi keeps 8 significant bits, q - hi is an
// integer below 2^7 in magnitude and so exact in bf16.
__device__ __forceinline__ void q_split8(const uint4& u, bf16x8& hi, bf16x8& lo) {
  const uint32_t wd[4] = {u.x, u.y, u.z, u.w};
  uint32_t h[4], l[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
    split2((float)(int)(int16_t)(wd[i] & 0xFFFFu), (float)((int)wd[i] >> 16), h[i], l[i]);
  hi = __builtin_bit_cast(bf16x8, make_uint4(h[0], h[1], h[2], h[3]));
  lo = __builtin_bit_cast(bf16x8, make_uint4(l[0], l[1], l[2], l[3]));
}
// Eight values (times the inverse scale) -> eight int16, nearest, saturated.
__device__ __forceinline__ uint4 q_pack8(const float (&x)[8], float inv) {
  const uint2 a = q_pack4(floatx4{x[0], x[1], x[2], x[3]}, inv);
  const uint2 b = q_pack4(floatx4{x[4], x[5], x[6], x[7]}, inv);
  return make_uint4(a.x, a.y, b.x, b.y);
}

// ---- transposed operand fragments from LDS --------------------------------
// ds_read_b64_tr_b16 (gfx950): inside each 16-lane group the 16 lanes' 8-byte
// reads form S[s][p] (lane s, element p), and lane i receives S[4e + i/4][i%4]
// for e = 0..3.  So when lane s of the group addresses row r0 + s/4, columns
// c0 + 4 (s%4) .. +3 of a row-major bf16 tile, lane i receives the column
// c0 + i at rows r0 .. r0 + 3: an MFMA operand fragment whose reduction index
// runs down the tile's rows.  (Layout established by an in-bounds probe.)
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ bf16x4_t ld_tr4(const bf16_t* tile, int ld, int r0, int c0) {
  const int s = lane_id() & 15;
  const bf16_t* p = tile + (r0 + (s >> 2)) * ld + c0 + 4 * (s & 3);
  const i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4*)(p));
  return __builtin_bit_cast(bf16x4_t, v);
}
// Eight consecutive rows r0 .. r0 + 7 of column c0 + (lane % 16).
__device__ __forceinline__ bf16x8 ld_tr8(const bf16_t* tile, int ld, int r0, int c0) {
  const bf16x4_t a = ld_tr4(tile, ld, r0, c0), b = ld_tr4(tile, ld, r0 + 4, c0);
  return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}

// ---- cross-lane reductions and scans (DPP: VALU only, no LDS round trip) ----
// DPP controls used (gfx9 encodings; a "row" is 16 lanes): quad_perm xor 1 /
// xor 2, row_half_mirror (lane i of an 8-lane half reads lane 7 - i), row_mirror
// (lane i reads 15 - i), row_shr:n (lane i reads i - n inside its row, old value
// at the row start), row_bcast15 / row_bcast31 (last lane of a row, resp. of
// the lower half, to the following rows selected by the row mask), wave_shl:1
// (lane i reads lane i + 1).  Directions were checked with an in-bounds probe.
template <int CTRL, int ROWMASK = 0xF>
__device__ __forceinline__ float dpp_upd(float old, float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, old),
                                                               __builtin_bit_cast(int, x), CTRL,
                                                               ROWMASK, 0xF, false));
}
// Sum over each group of 8 lanes (every lane of the group gets the same value).
__device__ __forceinline__ float sum8(float x) {
  x += dpp_upd<0xB1>(0.f, x);   // quad_perm [1,0,3,2]
  x += dpp_upd<0x4E>(0.f, x);   // quad_perm [2,3,0,1]
  x += dpp_upd<0x141>(0.f, x);  // row_half_mirror
  return x;
}
// Sum over the 16 lanes that hold one accumulator row (same lane / 16 group);
// a symmetric butterfly, so every lane of the row gets the same value.
__device__ __forceinline__ float sum16(float x) {
  x = sum8(x);
  x += dpp_upd<0x140>(0.f, x);  // row_mirror
  return x;
}
// Sum over the 4 lane groups (lanes l, l^16, l^32, l^48), every lane gets the
// result: v_permlane16_swap / v_permlane32_swap with both operands x hand lane l
// the values of lanes l & ~16 and l | 16 (resp. 32), VALU only.
__device__ __forceinline__ float sum_groups(float x) {
  const unsigned u = __float_as_uint(x);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const float y = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const unsigned v = __float_as_uint(y);
  const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}
// Value of `lane` (the readlane builtin moves 32-bit integers).
__device__ __forceinline__ float read_lane(float x, int lane) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), lane));
}
// Sum over the wavefront, uniform result.
__device__ __forceinline__ float wave_sum(float x) {
  x = sum16(x);
  return (read_lane(x, 0) + read_lane(x, 16)) + (read_lane(x, 32) + read_lane(x, 48));
}
// Value of lane + 1 (0 for the last lane).
__device__ __forceinline__ float shift_down1(float x) { return dpp_upd<0x130>(0.f, x); }
// Max over each group of 8 lanes, resp. the 16 lanes of a row (symmetric
// butterflies, every lane gets the result).
// (NaN-propagating, see nmax.)
__device__ __forceinline__ float max8(float m) {
  m = nmax(m, dpp_upd<0xB1>(0.f, m));   // quad_perm [1,0,3,2]
  m = nmax(m, dpp_upd<0x4E>(0.f, m));   // quad_perm [2,3,0,1]
  m = nmax(m, dpp_upd<0x141>(0.f, m));  // row_half_mirror
  return m;
}
__device__ __forceinline__ float max16(float m) {
  m = max8(m);
  return nmax(m, dpp_upd<0x140>(0.f, m));  // row_mirror
}
// Max over lanes l, l ^ 4, l ^ 8, l ^ 12 (the four lanes that hold one row
// after quad_transpose), every one of them gets the result.
__device__ __forceinline__ float row4_max(float m) {
  m = nmax(m, dpp_upd<0x124>(0.f, m));  // row_ror:4
  m = nmax(m, dpp_upd<0x128>(0.f, m));  // row_ror:8
  return m;
}

// ---- global -> register -> LDS tile copies ---------------------------------

// A NROWS x COLS tile of T held in registers, 16 bytes per slot, slots spread
// over the workgroup's threads.  load() issues every global load of the tile
// back to back (rows >= `rows` read as zero) so their latencies overlap; the
// store functions then write LDS.  Keeping load() and store() apart lets a
// kernel issue the next chunk's loads before computing on the current one.
template <typename T, int NROWS, int COLS, int NTHR = comba::NTHR>
struct TileRegs {
  static constexpr int V = 16 / sizeof(T);
  static constexpr int PER_ROW = COLS / V;
  static constexpr int TOTAL = NROWS * PER_ROW;
  static constexpr int ITER = (TOTAL + NTHR - 1) / NTHR;
  static_assert(COLS % V == 0, "tile rows must be whole 16-byte units");
  uint4 r[ITER];

  __device__ __forceinline__ void load(const T* __restrict__ g, long gs, int rows) {
#pragma unroll
    for (int it = 0; it < ITER; ++it) {
      const int idx = threadIdx.x + it * NTHR;
      const int rr = idx / PER_ROW, cc = (idx % PER_ROW) * V;
      uint4 val = make_uint4(0, 0, 0, 0);
      if ((TOTAL % NTHR == 0 || idx < TOTAL) && rr < rows)
        val = *reinterpret_cast<const uint4*>(g + (long)rr * gs + cc);
      r[it] = val;
    }
  }
  // The same tile through raw buffer loads whose record count ends at row
  // rows - 1: the hardware returns zeros past it, so there is no per-row branch
  // (a branch around a load leaves a copy of its result that waits for it at
  // once).  g is 4-byte aligned; the tile's byte extent fits in 32 bits.
  __device__ __forceinline__ void load_clip(const T* __restrict__ g, long gs, int rows) {
    const int nbytes = rows > 0 ? (int)(((long)(rows - 1) * gs + COLS) * (long)sizeof(T)) : 0;
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(g), 0, nbytes, 0x00020000);
#pragma unroll
    for (int it = 0; it < ITER; ++it) {
      const int idx = threadIdx.x + it * NTHR;
      const int rr = idx / PER_ROW, cc = (idx % PER_ROW) * V;
      // rows at or past NROWS (idx >= TOTAL) fall past the record count too (gs >= COLS)
      const unsigned off = (unsigned)(((long)rr * gs + cc) * (long)sizeof(T));
      r[it] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
    }
  }
  __device__ __forceinline__ void store(T* s, int ld) const {
#pragma unroll
    for (int it = 0; it < ITER; ++it) {
      const int idx = threadIdx.x + it * NTHR;
      if (TOTAL % NTHR == 0 || idx < TOTAL) {
        const int rr = idx / PER_ROW, cc = (idx % PER_ROW) * V;
        *reinterpret_cast<uint4*>(s + rr * ld + cc) = r[it];
      }
    }
  }
  // st[c * ldt + r] = tile[r][c]
  __device__ __forceinline__ void store_t(T* st, int ldt) const {
#pragma unroll
    for (int it = 0; it < ITER; ++it) {
      const int idx = threadIdx.x + it * NTHR;
      if (TOTAL % NTHR == 0 || idx < TOTAL) {
        const int rr = idx / PER_ROW, cc = (idx % PER_ROW) * V;
        union { uint4 u; T e[V]; } val;
        val.u = r[it];
#pragma unroll
        for (int e = 0; e < V; ++e) st[(cc + e) * ldt + rr] = val.e[e];
      }
    }
  }
};

// One-shot copies (load then store) for tiles that are not prefetched.
template <typename T, int NROWS, int COLS>
__device__ __forceinline__ void tile_to_lds(const T* __restrict__ g, long gs, int rows, T* s, int ld) {
  TileRegs<T, NROWS, COLS> t;
  t.load(g, gs, rows);
  t.store(s, ld);
}

// Inclusive prefix sum across the 64 lanes of a wavefront: within each row by
// shifts of 1, 2, 4, 8, then the row totals carried upward by row broadcasts.
__device__ __forceinline__ float wave_prefix_sum(float x) {
  x += dpp_upd<0x111>(0.f, x);       // row_shr:1
  x += dpp_upd<0x112>(0.f, x);       // row_shr:2
  x += dpp_upd<0x114>(0.f, x);       // row_shr:4
  x += dpp_upd<0x118>(0.f, x);       // row_shr:8
  x += dpp_upd<0x142, 0xA>(0.f, x);  // row_bcast15 into rows 1, 3
  x += dpp_upd<0x143, 0xC>(0.f, x);  // row_bcast31 into rows 2, 3
  return x;
}

}  // namespace comba
