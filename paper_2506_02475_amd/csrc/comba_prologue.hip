// Input prologue of the Comba layer (Section 3.4, Neural Architecture): the
// projected q, k, v pre-activations pass through a short causal depthwise
// convolution (K = 4 taps per channel, zero history at each sequence start),
// the SiLU feature map and, for q and k, an L2 normalisation over the head's
// channels; the results are the chunk operator's inputs.
//
//   u_t = sum_j w[j] x_{t-3+j},   s_t = u_t sigmoid(u_t),   y_t = s_t / sqrt(|s_t|^2 + eps)
//
// Both directions are streaming: one wavefront walks a run of 64 tokens of one
// head along the sequence, its lanes holding D / 64 consecutive channels each,
// with the convolution window in registers (every x row is read once, plus a
// three-row halo per run).  The L2 norms are wave reductions.
#include "comba_device.hpp"
#include "comba_launch.h"

namespace comba {

constexpr int PRO_RUN = 64;   // tokens per wave (backward; forward: fwd_run_tokens)
constexpr int PRO_K = 4;      // taps
constexpr int PRO_WAVES = 4;  // waves (runs) per workgroup
constexpr int PRO_PF = 8;     // token rows loaded ahead, together

template <typename Tin, int C>
__device__ __forceinline__ void load_ch(const Tin* p, float (&v)[C]) {
  if constexpr (is_f32<Tin>::value) {
    if constexpr (C == 1) {
      v[0] = *p;
    } else if constexpr (C == 2) {
      const float2 f = *reinterpret_cast<const float2*>(p);
      v[0] = f.x;
      v[1] = f.y;
    } else {
      const float4 f = *reinterpret_cast<const float4*>(p);
      v[0] = f.x;
      v[1] = f.y;
      v[2] = f.z;
      v[3] = f.w;
    }
  } else if constexpr (C == 1) {
    v[0] = bf2f(*p);
  } else if constexpr (C == 2) {
    const uint32_t u = *reinterpret_cast<const uint32_t*>(p);
    v[0] = __uint_as_float(u << 16);
    v[1] = __uint_as_float(u & 0xFFFF0000u);
  } else {
    static_assert(C == 4, "channels per lane");
    const uint2 u = *reinterpret_cast<const uint2*>(p);
    v[0] = __uint_as_float(u.x << 16);
    v[1] = __uint_as_float(u.x & 0xFFFF0000u);
    v[2] = __uint_as_float(u.y << 16);
    v[3] = __uint_as_float(u.y & 0xFFFF0000u);
  }
}

// Round to nearest even with the hardware conversion (v_cvt_pk_bf16_f32),
// which keeps NaN a NaN and Inf an Inf (adding a rounding bias to the bit
// pattern would turn a NaN with a full payload into -0).
__device__ __forceinline__ bf16_t f2bf(float x) {
  return __builtin_bit_cast(bf16_t, (__bf16)x);
}

// One vector store per lane and row (element-wise stores would leave every
// instruction writing only parts of each 4-byte word).
template <int C>
__device__ __forceinline__ void store_f32(float* p, const float (&v)[C]) {
  if constexpr (C == 1) {
    *p = v[0];
  } else if constexpr (C == 2) {
    *reinterpret_cast<float2*>(p) = make_float2(v[0], v[1]);
  } else {
    static_assert(C == 4, "channels per lane");
    *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  }
}

template <typename Tin, int C>
__device__ __forceinline__ void store_ch(Tin* p, const float (&v)[C]) {
  if constexpr (is_f32<Tin>::value) {
    store_f32<C>(p, v);
  } else if constexpr (C == 1) {
    *p = f2bf(v[0]);
  } else if constexpr (C == 2) {
    *reinterpret_cast<uint32_t*>(p) = (uint32_t)f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16);
  } else {
    *reinterpret_cast<uint2*>(p) = make_uint2((uint32_t)f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16),
                                              (uint32_t)f2bf(v[2]) | ((uint32_t)f2bf(v[3]) << 16));
  }
}

// Logistic function: the hardware reciprocal (v_rcp_f32, about 1 ulp) instead of
// an IEEE division, which costs ten instructions per element here.  1 + e^-u >= 1,
// so no denormal operand; u = -inf gives 0, u = +inf 1, NaN stays NaN.
__device__ __forceinline__ float sigm(float u) { return __builtin_amdgcn_rcpf(1.f + __expf(-u)); }

// Sequence [sa, se) holding token t.
__device__ __forceinline__ void seq_bounds(const int32_t* __restrict__ cu, int N, int Tseq, int Ttot,
                                           int t, int& sa, int& se) {
  if (!cu || N <= 0) {  // (the host rejects tokens without sequences)
    sa = cu ? 0 : (t / Tseq) * Tseq;
    se = cu ? Ttot : sa + Tseq;
    return;
  }
  // largest s < N with cu[s] <= t (then cu[s + 1] > t: empty sequences skipped)
  int lo = 0, hi = N - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cu[mid] <= t) lo = mid; else hi = mid - 1;
  }
  sa = min(max(cu[lo], 0), t);
  se = min(max(cu[lo + 1], t + 1), Ttot);
}

// Forward.  A wave takes one run of tokens (fwd_run_tokens) of 64 / (D / C) consecutive
// heads: each lane holds C consecutive channels of one head, so the rows of a
// token for those heads (contiguous in the [token][head][channel] layout)
// arrive as one 2C-byte load per lane (bf16), and a head's norm is a sum over
// its D / C lanes (DPP inside a row, no wave-wide reduction).
constexpr int PRO_FCL = 4;  // channels per lane
constexpr int PRO_FPF = 8;  // token rows per block

template <int LPR>
__device__ __forceinline__ float sum_lanes(float x) {
  if constexpr (LPR == 8) {
    return sum8(x);
  } else if constexpr (LPR == 16) {
    return sum16(x);
  } else if constexpr (LPR == 32) {
    x = sum16(x);
    return x + __shfl_xor(x, 16);
  } else {
    static_assert(LPR == 64, "lanes per head row");
    return wave_sum(x);
  }
}

// C channels of one row as loaded (4-byte words, 8 or 16 bytes per load).
template <typename Tin, int C>
struct RowC {
  static constexpr int W = C * (int)sizeof(Tin) / 4;
  static_assert(W == 2 || W % 4 == 0, "row piece of 8 or 16k bytes");
  uint32_t r[W];
  __device__ __forceinline__ void load(const Tin* p) {
    if constexpr (W == 2) {
      const uint2 u = *reinterpret_cast<const uint2*>(p);
      r[0] = u.x;
      r[1] = u.y;
    } else {
#pragma unroll
      for (int i = 0; i < W / 4; ++i) {
        const uint4 u = reinterpret_cast<const uint4*>(p)[i];
        r[4 * i] = u.x;
        r[4 * i + 1] = u.y;
        r[4 * i + 2] = u.z;
        r[4 * i + 3] = u.w;
      }
    }
  }
  __device__ __forceinline__ void unpack(float (&v)[C]) const {
    if constexpr (is_f32<Tin>::value) {
#pragma unroll
      for (int i = 0; i < C; ++i) v[i] = __uint_as_float(r[i]);
    } else {
#pragma unroll
      for (int i = 0; i < W; ++i) {
        v[2 * i] = __uint_as_float(r[i] << 16);
        v[2 * i + 1] = __uint_as_float(r[i] & 0xFFFF0000u);
      }
    }
  }
};

template <typename Tin, int C>
__device__ __forceinline__ void store_rowc(Tin* p, const float (&v)[C]) {
  if constexpr (is_f32<Tin>::value) {
#pragma unroll
    for (int i = 0; i < C / 4; ++i)
      reinterpret_cast<float4*>(p)[i] = make_float4(v[4 * i], v[4 * i + 1], v[4 * i + 2], v[4 * i + 3]);
  } else {
    uint32_t u[C / 2];
#pragma unroll
    for (int i = 0; i < C / 2; ++i) u[i] = (uint32_t)f2bf(v[2 * i]) | ((uint32_t)f2bf(v[2 * i + 1]) << 16);
    if constexpr (C == 4) {
      *reinterpret_cast<uint2*>(p) = make_uint2(u[0], u[1]);
    } else {
#pragma unroll
      for (int i = 0; i < C / 8; ++i)
        reinterpret_cast<uint4*>(p)[i] = make_uint4(u[4 * i], u[4 * i + 1], u[4 * i + 2], u[4 * i + 3]);
    }
  }
}

template <typename Tin, int D, bool NORM>
__device__ __forceinline__ void prologue_fwd_run(const Tin* __restrict__ x, const float* __restrict__ w,
                                                 Tin* __restrict__ y, const int32_t* __restrict__ cu,
                                                 int N, int Tseq, int Ttot, int H, int run, int rlen,
                                                 int hgrp, float eps) {
  constexpr int C = PRO_FCL, PF = PRO_FPF, LPR = D / C, HPW = 64 / LPR;
  const int lane = lane_id();
  const int t0 = run * rlen, t1 = min(t0 + rlen, Ttot);
  if (t0 >= Ttot || hgrp * HPW >= H) return;  // wave-uniform
  const int h = hgrp * HPW + lane / LPR;
  const bool hv = h < H;  // lanes of heads past H compute on head H - 1 and store nothing
  const long ts = (long)H * D;  // token stride
  const long hoff = (long)min(h, H - 1) * D + (lane % LPR) * C;
  float wt[C][PRO_K];  // (w is only 4-byte aligned)
#pragma unroll
  for (int i = 0; i < C; ++i)
#pragma unroll
    for (int j = 0; j < PRO_K; ++j) wt[i][j] = w[(hoff + i) * PRO_K + j];
  int sa, se;
  seq_bounds(cu, N, Tseq, Ttot, t0, sa, se);
  // window: x of tokens t-3, t-2, t-1 (zero before the sequence start)
  float xw[PRO_K - 1][C];
#pragma unroll
  for (int m = 0; m < PRO_K - 1; ++m) {
    const int tt = t0 - (PRO_K - 1) + m;
    if (tt >= sa) {
      RowC<Tin, C> r;
      r.load(x + tt * ts + hoff);
      r.unpack(xw[m]);
    } else {
#pragma unroll
      for (int i = 0; i < C; ++i) xw[m][i] = 0.f;
    }
  }
  RowC<Tin, C> xr[PF];
#pragma unroll
  for (int e = 0; e < PF; ++e) xr[e].load(x + min(t0 + e, t1 - 1) * ts + hoff);
  for (int tb = t0; tb < t1; tb += PF) {
    // the next block's rows are in flight while this block is computed and
    // stored (issued before this block's stores, so waiting for them later
    // does not wait for those stores)
    RowC<Tin, C> xn[PF];
    if (tb + PF < t1) {
#pragma unroll
      for (int e = 0; e < PF; ++e) xn[e].load(x + min(tb + PF + e, t1 - 1) * ts + hoff);
    } else {
#pragma unroll
      for (int e = 0; e < PF; ++e)
#pragma unroll
        for (int i = 0; i < RowC<Tin, C>::W; ++i) xn[e].r[i] = 0u;
    }
    if (tb + PF <= t1 && tb + PF <= se) {
      // the block lies inside one sequence (the usual case): straight-line
      // code, so the tokens' independent norm reductions overlap
      float hx[PRO_K - 1 + PF][C], sv[PF][C], ssv[PF];
#pragma unroll
      for (int m = 0; m < PRO_K - 1; ++m)
#pragma unroll
        for (int i = 0; i < C; ++i) hx[m][i] = xw[m][i];
#pragma unroll
      for (int e = 0; e < PF; ++e) xr[e].unpack(hx[PRO_K - 1 + e]);
#pragma unroll
      for (int e = 0; e < PF; ++e) {
        ssv[e] = 0.f;
#pragma unroll
        for (int i = 0; i < C; ++i) {
          float u = wt[i][PRO_K - 1] * hx[e + PRO_K - 1][i];
#pragma unroll
          for (int m = 0; m < PRO_K - 1; ++m) u = fmaf(wt[i][m], hx[e + m][i], u);
          sv[e][i] = u * sigm(u);
          ssv[e] = fmaf(sv[e][i], sv[e][i], ssv[e]);
        }
      }
#pragma unroll
      for (int e = 0; e < PF; ++e) {
        if constexpr (NORM) {
          const float inv = rsqrtf(sum_lanes<LPR>(ssv[e]) + eps);
#pragma unroll
          for (int i = 0; i < C; ++i) sv[e][i] *= inv;
        }
        if (hv) store_rowc<Tin, C>(y + (tb + e) * ts + hoff, sv[e]);
      }
#pragma unroll
      for (int m = 0; m < PRO_K - 1; ++m)
#pragma unroll
        for (int i = 0; i < C; ++i) xw[m][i] = hx[PF + m][i];
    } else {
#pragma unroll
    for (int e = 0; e < PF; ++e) {
      const int t = tb + e;
      if (t >= t1) break;
      if (t >= se) {  // next (non-empty) sequence: no history
        seq_bounds(cu, N, Tseq, Ttot, t, sa, se);
#pragma unroll
        for (int m = 0; m < PRO_K - 1; ++m)
#pragma unroll
          for (int i = 0; i < C; ++i) xw[m][i] = 0.f;
      }
      float xt[C], s[C];
      xr[e].unpack(xt);
      float ss = 0.f;
#pragma unroll
      for (int i = 0; i < C; ++i) {
        float u = wt[i][PRO_K - 1] * xt[i];
#pragma unroll
        for (int m = 0; m < PRO_K - 1; ++m) u = fmaf(wt[i][m], xw[m][i], u);
        s[i] = u * sigm(u);
        ss = fmaf(s[i], s[i], ss);
      }
      if constexpr (NORM) {
        const float inv = rsqrtf(sum_lanes<LPR>(ss) + eps);
#pragma unroll
        for (int i = 0; i < C; ++i) s[i] *= inv;
      }
      if (hv) store_rowc<Tin, C>(y + t * ts + hoff, s);
#pragma unroll
      for (int i = 0; i < C; ++i) {
#pragma unroll
        for (int m = 0; m < PRO_K - 2; ++m) xw[m][i] = xw[m + 1][i];
        xw[PRO_K - 2][i] = xt[i];
      }
    }
    }
#pragma unroll
    for (int e = 0; e < PF; ++e) xr[e] = xn[e];
  }
}

// Head groups of the forward grid: enough for the tensor with the most.
template <int DK, int DV>
constexpr int fwd_head_groups(int H) {
  constexpr int D = DK > DV ? DK : DV, HPW = 64 / (D / PRO_FCL);
  return (H + HPW - 1) / HPW;
}

template <typename Tin, int DK, int DV>
__global__ __launch_bounds__(64 * PRO_WAVES) void k_prologue_fwd(PrologueArgs a) {
  const int run = blockIdx.x * PRO_WAVES + wave_id_s();
  const int z = blockIdx.z, hg = blockIdx.y;
  if (z == 0)
    prologue_fwd_run<Tin, DK, true>(static_cast<const Tin*>(a.xq), a.wq, static_cast<Tin*>(a.q),
                                    a.cu_seqlens, a.N, a.Tseq, a.Ttot, a.H, run, a.frun, hg, a.eps);
  else if (z == 1)
    prologue_fwd_run<Tin, DK, true>(static_cast<const Tin*>(a.xk), a.wk, static_cast<Tin*>(a.k),
                                    a.cu_seqlens, a.N, a.Tseq, a.Ttot, a.H, run, a.frun, hg, a.eps);
  else
    prologue_fwd_run<Tin, DV, false>(static_cast<const Tin*>(a.xv), a.wv, static_cast<Tin*>(a.v),
                                     a.cu_seqlens, a.N, a.Tseq, a.Ttot, a.H, run, a.frun, hg, a.eps);
}

// Backward of one run: dx rows [t0, t1) and this run's share of dw.  du is
// formed for tokens [t0, t1 + 3) (the last three belong to the next run but
// feed this run's last rows); du_t adds w[j] du_t to dx row t - 3 + j, kept in
// a four-row register accumulator whose oldest row is complete after each token.
// As in the forward, a wave takes 64 / (D / C) consecutive heads, C channels
// per lane (C = PRO_BCL: 16-byte gradient rows per lane).
constexpr int PRO_BCL = 4;

template <typename Tin, int D, bool NORM>
__device__ __forceinline__ void prologue_bwd_run(const Tin* __restrict__ x, const float* __restrict__ w,
                                                 const float* __restrict__ dy, float* __restrict__ dx,
                                                 float4* dwl, const int32_t* __restrict__ cu,
                                                 int N, int Tseq, int Ttot, int H, int run, int hgrp,
                                                 float eps) {
  constexpr int C = PRO_BCL, LPR = D / C, HPW = 64 / LPR;
  const int lane = lane_id();
  const int t0 = run * PRO_RUN, t1 = min(t0 + PRO_RUN, Ttot);
  // this wave's share of dw: slot lane * C + i = (head in group) * D + channel
  if (t0 >= Ttot || hgrp * HPW >= H) {  // no run: a zero share
#pragma unroll
    for (int i = 0; i < C; ++i) dwl[lane * C + i] = make_float4(0.f, 0.f, 0.f, 0.f);
    return;
  }
  const int h = hgrp * HPW + lane / LPR;
  const bool hv = h < H;  // lanes of heads past H compute on head H - 1 and store nothing
  const long ts = (long)H * D;
  const long hoff = (long)min(h, H - 1) * D + (lane % LPR) * C;
  float wt[C][PRO_K], dw[C][PRO_K];
#pragma unroll
  for (int i = 0; i < C; ++i)
#pragma unroll
    for (int j = 0; j < PRO_K; ++j) {
      wt[i][j] = w[(hoff + i) * PRO_K + j];
      dw[i][j] = 0.f;
    }
  int sa, se;
  seq_bounds(cu, N, Tseq, Ttot, t0, sa, se);
  float xw[PRO_K - 1][C], acc[PRO_K][C];  // acc[m]: dx row t - 3 + m
#pragma unroll
  for (int m = 0; m < PRO_K - 1; ++m) {
    const int tt = t0 - (PRO_K - 1) + m;
    if (tt >= sa) {
      load_ch<Tin, C>(x + tt * ts + hoff, xw[m]);
    } else {
#pragma unroll
      for (int i = 0; i < C; ++i) xw[m][i] = 0.f;
    }
  }
#pragma unroll
  for (int m = 0; m < PRO_K; ++m)
#pragma unroll
    for (int i = 0; i < C; ++i) acc[m][i] = 0.f;
  // store the pending rows t-3 .. t-3+cnt-1 that are this run's and in the sequence
  auto flush = [&](int t, int cnt) {
#pragma unroll
    for (int m = 0; m < PRO_K - 1; ++m) {
      const int r = t - (PRO_K - 1) + m;
      if (hv && m < cnt && r >= t0 && r < t1 && r >= sa) store_f32<C>(dx + r * ts + hoff, acc[m]);
    }
  };
  const int tstop = min(t1 + PRO_K - 1, Ttot);
  bool done = false;
  for (int tb = t0; tb < tstop && !done; tb += PRO_PF) {
  float xb[PRO_PF][C], gb[PRO_PF][C];
#pragma unroll
  for (int e = 0; e < PRO_PF; ++e) {
    const long row = min(tb + e, tstop - 1) * ts + hoff;
    load_ch<Tin, C>(x + row, xb[e]);
    load_ch<float, C>(dy + row, gb[e]);
  }
#pragma unroll
  for (int e = 0; e < PRO_PF; ++e) {
    const int t = tb + e;
    if (t >= tstop) break;
    if (t >= se) {
      // sequence end: its last rows are complete
      flush(t, PRO_K - 1);
      if (t >= t1) {  // the rest belongs to later runs
        done = true;
        break;
      }
      seq_bounds(cu, N, Tseq, Ttot, t, sa, se);
#pragma unroll
      for (int m = 0; m < PRO_K; ++m)
#pragma unroll
        for (int i = 0; i < C; ++i) acc[m][i] = 0.f;
#pragma unroll
      for (int m = 0; m < PRO_K - 1; ++m)
#pragma unroll
        for (int i = 0; i < C; ++i) xw[m][i] = 0.f;
    }
    float u[C], sg[C], s[C];
    const float (&xt)[C] = xb[e];
    const float (&g)[C] = gb[e];
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < C; ++i) {
      float uu = wt[i][PRO_K - 1] * xt[i];
#pragma unroll
      for (int m = 0; m < PRO_K - 1; ++m) uu = fmaf(wt[i][m], xw[m][i], uu);
      u[i] = uu;
      sg[i] = sigm(uu);
      s[i] = uu * sg[i];
      ss = fmaf(s[i], s[i], ss);
    }
    float ds[C];
    if constexpr (NORM) {
      const float inv = rsqrtf(sum_lanes<LPR>(ss) + eps);
      float yg = 0.f;
#pragma unroll
      for (int i = 0; i < C; ++i) yg = fmaf(s[i] * inv, g[i], yg);
      yg = sum_lanes<LPR>(yg);
#pragma unroll
      for (int i = 0; i < C; ++i) ds[i] = (g[i] - s[i] * inv * yg) * inv;
    } else {
#pragma unroll
      for (int i = 0; i < C; ++i) ds[i] = g[i];
    }
    const bool own = t < t1;
#pragma unroll
    for (int i = 0; i < C; ++i) {
      const float du = ds[i] * sg[i] * (1.f + u[i] * (1.f - sg[i]));
#pragma unroll
      for (int j = 0; j < PRO_K; ++j) acc[j][i] = fmaf(wt[i][j], du, acc[j][i]);
      if (own) {
#pragma unroll
        for (int j = 0; j < PRO_K - 1; ++j) dw[i][j] = fmaf(du, xw[j][i], dw[i][j]);
        dw[i][PRO_K - 1] = fmaf(du, xt[i], dw[i][PRO_K - 1]);
      }
    }
    // row t - 3 has all its terms
    {
      const int r = t - (PRO_K - 1);
      if (hv && r >= t0 && r < t1 && r >= sa) store_f32<C>(dx + r * ts + hoff, acc[0]);
    }
#pragma unroll
    for (int i = 0; i < C; ++i) {
#pragma unroll
      for (int m = 0; m < PRO_K - 1; ++m) acc[m][i] = acc[m + 1][i];
      acc[PRO_K - 1][i] = 0.f;
#pragma unroll
      for (int m = 0; m < PRO_K - 2; ++m) xw[m][i] = xw[m + 1][i];
      xw[PRO_K - 2][i] = xt[i];
    }
  }
  }
  // the walk ended at t1 + 3 or at the end of the tokens (then flush here), or
  // at a sequence end past t1 (flushed there): every pending row is complete
  if (!done) flush(tstop, PRO_K - 1);
  // this run's share of dw, combined with the other waves' in LDS
#pragma unroll
  for (int i = 0; i < C; ++i) dwl[lane * C + i] = make_float4(dw[i][0], dw[i][1], dw[i][2], dw[i][3]);
}

// Sum of the workgroup's wave shares of dw (fixed order) into its partial
// [block][h][D] (four taps per float4), for the heads of its group.
template <int D>
__device__ __forceinline__ void combine_dw(const float4 (*dws)[256], float* __restrict__ dwp, int H) {
  constexpr int HPW = 64 / (D / PRO_BCL);
  const int h0 = blockIdx.y * HPW;
  float4* out = reinterpret_cast<float4*>(dwp) + ((long)blockIdx.x * H + h0) * D;
  const int n = min(HPW, H - h0) * D;  // slots of existing heads (n <= 0: none)
  for (int c = threadIdx.x; c < n; c += 64 * PRO_WAVES) {
    float4 s = dws[0][c];
#pragma unroll
    for (int w = 1; w < PRO_WAVES; ++w) {
      const float4 v = dws[w][c];
      s = make_float4(s.x + v.x, s.y + v.y, s.z + v.z, s.w + v.w);
    }
    out[c] = s;
  }
}

template <typename Tin, int DK, int DV>
__global__ __launch_bounds__(64 * PRO_WAVES) void k_prologue_bwd(PrologueArgs a) {
  static_assert(64 * PRO_BCL <= 256, "slots per wave share");
  __shared__ float4 dws[PRO_WAVES][256];  // per wave: the four tap sums of each channel
  // every wave reaches the barrier below (runs past the tokens add zeros)
  const int run = blockIdx.x * PRO_WAVES + wave_id_s();
  const int z = blockIdx.z;
  float4* dwl = dws[wave_id_s()];
  if (z == 0)
    prologue_bwd_run<Tin, DK, true>(static_cast<const Tin*>(a.xq), a.wq, a.gq, a.dxq, dwl,
                                    a.cu_seqlens, a.N, a.Tseq, a.Ttot, a.H, run, blockIdx.y, a.eps);
  else if (z == 1)
    prologue_bwd_run<Tin, DK, true>(static_cast<const Tin*>(a.xk), a.wk, a.gk, a.dxk, dwl,
                                    a.cu_seqlens, a.N, a.Tseq, a.Ttot, a.H, run, blockIdx.y, a.eps);
  else
    prologue_bwd_run<Tin, DV, false>(static_cast<const Tin*>(a.xv), a.wv, a.gv, a.dxv, dwl,
                                     a.cu_seqlens, a.N, a.Tseq, a.Ttot, a.H, run, blockIdx.y, a.eps);
  __syncthreads();
  if (z == 0) combine_dw<DK>(dws, a.dwpq, a.H);
  else if (z == 1) combine_dw<DK>(dws, a.dwpk, a.H);
  else combine_dw<DV>(dws, a.dwpv, a.H);
}

// Head groups of the backward grid: enough for the tensor with the most.
template <int DK, int DV>
constexpr int bwd_head_groups(int H) {
  constexpr int D = DK > DV ? DK : DV, HPW = 64 / (D / PRO_BCL);
  return (H + HPW - 1) / HPW;
}

// dw[i] = sum over the workgroups' partials (fixed order), for q, k and v.
__global__ __launch_bounds__(256) void k_prologue_dw(PrologueArgs a) {
  const int z = blockIdx.y;
  const long n = (long)a.H * (z == 2 ? a.dv : a.dk) * PRO_K;
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const float* p = z == 0 ? a.dwpq : (z == 1 ? a.dwpk : a.dwpv);
  const int nblk = (a.nruns + PRO_WAVES - 1) / PRO_WAVES;
  float s = 0.f;
  for (int r = 0; r < nblk; ++r) s += p[(long)r * n + i];
  (z == 0 ? a.dwq : (z == 1 ? a.dwk : a.dwv))[i] = s;
}

// Tokens per forward run, a multiple of PRO_FPF.  The runs of all (head group,
// tensor) items are sized to fill the device's resident wave slots once: the
// waves all carry the same work, so a second, partial round would leave most
// of the device idle for a whole run.  (Fixed 64-token runs when the device
// cannot be queried.)
template <typename Tin, int DK, int DV>
static int fwd_run_tokens(int Ttot, int groups) {
  static const int slots = [] {
    int dev = 0, cus = 0, nb = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, k_prologue_fwd<Tin, DK, DV>,
                                                     64 * PRO_WAVES, 0) != hipSuccess)
      return 0;
    return cus * nb * PRO_WAVES;
  }();
  if (slots <= 0) return PRO_RUN;
  const int items = 3 * groups;
  const int per_item = slots > items ? slots / items : 1;
  const int run = (Ttot + per_item - 1) / per_item;
  return max(PRO_FPF, (run + PRO_FPF - 1) / PRO_FPF * PRO_FPF);
}

template <typename Tin, int DK, int DV>
static hipError_t run_prologue(const PrologueArgs& a, bool bwd) {
  const dim3 grid((a.nruns + PRO_WAVES - 1) / PRO_WAVES, a.H, 3);
  if (!bwd) {
    a.stage("prologue_fwd");
    PrologueArgs f = a;
    const int groups = fwd_head_groups<DK, DV>(a.H);
    f.frun = fwd_run_tokens<Tin, DK, DV>(a.Ttot, groups);
    const int fruns = (a.Ttot + f.frun - 1) / f.frun;
    const dim3 fgrid((fruns + PRO_WAVES - 1) / PRO_WAVES, groups, 3);
    if (fruns > 0) k_prologue_fwd<Tin, DK, DV><<<fgrid, 64 * PRO_WAVES, 0, a.stream>>>(f);
  } else {
    a.stage("prologue_bwd");
    const dim3 bgrid(grid.x, bwd_head_groups<DK, DV>(a.H), 3);
    if (a.nruns > 0) k_prologue_bwd<Tin, DK, DV><<<bgrid, 64 * PRO_WAVES, 0, a.stream>>>(a);
    a.stage("prologue_dw");
    const int dmax = a.dk > a.dv ? a.dk : a.dv;
    k_prologue_dw<<<dim3((a.H * dmax * PRO_K + 255) / 256, 3), 256, 0, a.stream>>>(a);
  }
  a.stage(nullptr);
  return hipGetLastError();
}

template <typename Tin>
static hipError_t dispatch_prologue(const PrologueArgs& a, bool bwd) {
  if (a.dk == 64 && a.dv == 64) return run_prologue<Tin, 64, 64>(a, bwd);
  if (a.dk == 64 && a.dv == 128) return run_prologue<Tin, 64, 128>(a, bwd);
  if (a.dk == 128 && a.dv == 64) return run_prologue<Tin, 128, 64>(a, bwd);
  if (a.dk == 128 && a.dv == 128) return run_prologue<Tin, 128, 128>(a, bwd);
  if (a.dk == 256 && a.dv == 256) return run_prologue<Tin, 256, 256>(a, bwd);
  if (a.dk == 128 && a.dv == 256) return run_prologue<Tin, 128, 256>(a, bwd);
  if (a.dk == 256 && a.dv == 128) return run_prologue<Tin, 256, 128>(a, bwd);
  return hipErrorInvalidValue;
}

// Output gate (Section 3.4, sigmoid gating): y = o sigmoid(z); backward
// do = dy sigmoid(z), dz = dy o sigmoid(z) (1 - sigmoid(z)).  Four elements per
// thread, elementwise over the whole [B, T, H, dv] tensor.
template <typename Tin>
__global__ __launch_bounds__(256) void k_gate(const float* __restrict__ o, const Tin* __restrict__ z,
                                              Tin* __restrict__ y, const float* __restrict__ dy,
                                              float* __restrict__ dout, float* __restrict__ dz,
                                              long n4) {
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i >= n4) return;
  float ov[4], zv[4], sg[4];
  load_ch<float, 4>(o + 4 * i, ov);
  load_ch<Tin, 4>(z + 4 * i, zv);
#pragma unroll
  for (int e = 0; e < 4; ++e) sg[e] = sigm(zv[e]);
  if (!dy) {
    float yv[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) yv[e] = ov[e] * sg[e];
    store_ch<Tin, 4>(y + 4 * i, yv);
  } else {
    float gv[4], a[4], b[4];
    load_ch<float, 4>(dy + 4 * i, gv);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      a[e] = gv[e] * sg[e];
      b[e] = a[e] * ov[e] * (1.f - sg[e]);
    }
    store_f32<4>(dout + 4 * i, a);
    store_f32<4>(dz + 4 * i, b);
  }
}

hipError_t launch_gate(bool bf16, long n, const float* o, const void* z, void* y, const float* dy,
                       float* dout, float* dz, hipStream_t st) {
  const long n4 = n / 4;
  if (n4 == 0) return hipSuccess;
  const dim3 grid((unsigned)((n4 + 255) / 256));
  if (bf16)
    k_gate<bf16_t><<<grid, 256, 0, st>>>(o, static_cast<const bf16_t*>(z), static_cast<bf16_t*>(y),
                                         dy, dout, dz, n4);
  else
    k_gate<float><<<grid, 256, 0, st>>>(o, static_cast<const float*>(z), static_cast<float*>(y), dy,
                                        dout, dz, n4);
  return hipGetLastError();
}

hipError_t launch_prologue(const PrologueArgs& a, bool bwd) {
  return a.bf16 ? dispatch_prologue<bf16_t>(a, bwd) : dispatch_prologue<float>(a, bwd);
}

}  // namespace comba
