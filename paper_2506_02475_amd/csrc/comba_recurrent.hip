// Recurrent (token-by-token) form of the Comba recurrence (Eq. comba-S, the
// constant-memory inference mode of Section 3): per sequence and head, with the
// state kept transposed as H = S^T (dk x dv),
//
//   a_t = H_{t-1}^T k_t                       (= S_{t-1} k_t)
//   u_t = beta_t v_t - beta~_t a_t
//   H_t = alpha_t H_{t-1} + k_t u_t^T
//   o_t = H_t^T (q_t - d k_t) = alpha_t H_{t-1}^T q~_t + u_t (k_t . q~_t)
//
// The last identity lets one pass over the state produce both reductions a_t
// and H_{t-1}^T q~_t before the update, so each token reads the state once (from
// registers) and the whole call reads and writes it in HBM exactly once.  For
// decoding (one token per sequence) the kernel is bound by those 2 x dk x dv x 4
// bytes of state traffic per head.
#include "comba_device.hpp"
#include "comba_launch.h"

namespace comba {

// Four consecutive values of a row as fp32.
__device__ __forceinline__ float4 load4f(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ float4 load4f(const bf16_t* p) {
  const uint2 u = *reinterpret_cast<const uint2*>(p);
  return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u),
                     __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xFFFF0000u));
}

// The states stream through once per call: nontemporal accesses keep them
// from displacing other data in the caches (and measure 17% faster on a
// decoding step than plain ones).
typedef float f32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ float4 load4_stream(const float* p) {
  const f32x4 x = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
  return make_float4(x[0], x[1], x[2], x[3]);
}
__device__ __forceinline__ void store4_stream(float* p, const float4& v) {
  const f32x4 x = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(x, reinterpret_cast<f32x4*>(p));
}

__device__ __forceinline__ float4 f4_fma(float s, const float4& x, const float4& y) {
  return make_float4(fmaf(s, x.x, y.x), fmaf(s, x.y, y.y), fmaf(s, x.z, y.z), fmaf(s, x.w, y.w));
}

// Sum of x over the lanes of a wave that hold the same column quad (lanes
// cq + QB r): every such lane gets the total.
template <int QB>
__device__ __forceinline__ float sum_rowgroups(float x) {
  static_assert(QB == 4 || QB == 8 || QB == 16 || QB == 32, "column quads per row slice");
  if constexpr (QB == 4) x += __shfl_xor(x, 4);
  if constexpr (QB <= 8) x += dpp_upd<0x128>(0.f, x);  // row_ror:8 (= lane ^ 8 inside a row)
  if constexpr (QB <= 16) x += __shfl_xor(x, 16);
  x += __shfl_xor(x, 32);
  return x;
}

// ---------------------------------------------------------------------------
// k_recurrent: one workgroup of NW waves per (sequence, head, BV-wide slice of
// dv; BV = dv at the usual shapes, so one workgroup owns a whole state).  Wave
// w owns the RW = dk / NW rows w RW ..; lane l of it the entries
// H[i][j0 + 4 cq .. 4 cq + 3] (cq = l % QB) of the rows i = w RW + rg + RGW m
// (rg = l / QB, m < RPT), held in registers for the whole sequence.  One load
// or store instruction of a wave thus covers RGW whole consecutive rows of the
// slice (1 KiB at dv = 128): the state streams through HBM in contiguous
// pieces.  Reductions over rows: lane shuffles inside a wave, then one LDS
// exchange between the waves.  The next token's inputs are loaded while the
// current one is processed.  h0 may be NULL (zero state) and ht NULL (not
// stored); ht may be the same buffer as h0 (each lane reads its entries before
// writing them).
// ---------------------------------------------------------------------------
template <typename Tin, int DK, int DV, int BV, int NW>
__global__ __launch_bounds__(64 * NW) void k_recurrent(
    const Tin* __restrict__ q, const Tin* __restrict__ k, const Tin* __restrict__ v,
    const float* __restrict__ g, const Tin* __restrict__ beta, const Tin* __restrict__ beta_tilde,
    const float* __restrict__ d, const int32_t* __restrict__ cu_seqlens, int Tseq, int Ttot, int H,
    const float* h0, float* __restrict__ o, float* ht) {
  constexpr int QB = BV / 4;     // column quads of the slice (lanes per row)
  constexpr int RGW = 64 / QB;   // rows covered by one wave instruction
  constexpr int RW = DK / NW;    // rows per wave
  constexpr int RPT = RW / RGW;  // rows per lane
  constexpr int KW = (DK + 63) / 64;  // waves that load one element of k, q each
  static_assert(RW % RGW == 0 && RPT % 4 == 0 && KW <= NW, "row split");
  // k and q~ in lane order: entry (w RGW + rg) RPT + m is row w RW + rg + RGW m,
  // so a lane reads its rows four at a time
  __shared__ __align__(16) float Ks[2][DK], Qs[2][DK];
  __shared__ float4 red[2][NW][QB][2];  // per wave: partial H^T k, H^T q~ of each column quad
  __shared__ float kqp[2][KW];          // per wave: partial k . q~

  const int s = blockIdx.x, h = blockIdx.y, j0 = blockIdx.z * BV;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int cq = lane % QB, rg = lane / QB;
  int t0, len;
  if (cu_seqlens) {
    // offsets outside [0, Ttot] or decreasing are clamped (never out of bounds)
    t0 = min(max(cu_seqlens[s], 0), Ttot);
    len = min(max(cu_seqlens[s + 1], t0), Ttot) - t0;
  } else {
    t0 = s * Tseq;
    len = Tseq;
  }
  const float dh = d[h];
  // this lane's first entry: row w RW + rg, columns j0 + 4 cq ..
  const long soff = ((long)s * H + h) * DK * DV + (long)(w * RW + rg) * DV + j0 + 4 * cq;
  const int lpos = (w * RGW + rg) * RPT;  // this lane's k, q~ entries in LDS
  // the LDS slot of row tid (rows tid < DK are loaded by thread tid)
  const int wr = tid / RW, rr = tid % RW;
  const int spos = (wr * RGW + rr % RGW) * RPT + rr / RGW;

  float4 hs[RPT];
#pragma unroll
  for (int m = 0; m < RPT; ++m)
    hs[m] = h0 ? load4_stream(h0 + soff + (long)RGW * m * DV) : make_float4(0.f, 0.f, 0.f, 0.f);

  float pk = 0.f, pq = 0.f, pg = 0.f, pb = 0.f, pbt = 0.f;
  float4 pv = make_float4(0.f, 0.f, 0.f, 0.f);
  auto load_token = [&](int t) {
    const long row = (long)(t0 + t) * H + h;
    if (tid < DK) {
      pk = to_f(k[row * DK + tid]);
      pq = to_f(q[row * DK + tid]);
    }
    pv = load4f(v + row * DV + j0 + 4 * cq);
    pg = g[row];
    pb = to_f(beta[row]);
    pbt = to_f(beta_tilde[row]);
  };
  if (len > 0) load_token(0);

  for (int t = 0; t < len; ++t) {
    // two buffers: a wave can only reach token t + 2's writes after every wave
    // has passed token t + 1's first barrier, i.e. finished reading token t
    const int buf = t & 1;
    const float kt = pk, qt = pq - dh * pk;
    const float4 vt = pv;
    const float alpha = __expf(pg), bt = pb, btt = pbt;
    if (tid < DK) {
      Ks[buf][spos] = kt;
      Qs[buf][spos] = qt;
    }
    if (w < KW) {
      const float x = wave_sum(tid < DK ? kt * qt : 0.f);
      if (lane == 0) kqp[buf][w] = x;
    }
    __syncthreads();
    if (t + 1 < len) load_token(t + 1);

    // partial H^T k and H^T q~ of this lane's columns over its rows
    float4 a = make_float4(0.f, 0.f, 0.f, 0.f), b = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int m = 0; m < RPT; m += 4) {
      const float4 k4 = *reinterpret_cast<const float4*>(&Ks[buf][lpos + m]);
      const float4 q4 = *reinterpret_cast<const float4*>(&Qs[buf][lpos + m]);
      a = f4_fma(k4.x, hs[m], a);
      a = f4_fma(k4.y, hs[m + 1], a);
      a = f4_fma(k4.z, hs[m + 2], a);
      a = f4_fma(k4.w, hs[m + 3], a);
      b = f4_fma(q4.x, hs[m], b);
      b = f4_fma(q4.y, hs[m + 1], b);
      b = f4_fma(q4.z, hs[m + 2], b);
      b = f4_fma(q4.w, hs[m + 3], b);
    }
    a.x = sum_rowgroups<QB>(a.x);
    a.y = sum_rowgroups<QB>(a.y);
    a.z = sum_rowgroups<QB>(a.z);
    a.w = sum_rowgroups<QB>(a.w);
    b.x = sum_rowgroups<QB>(b.x);
    b.y = sum_rowgroups<QB>(b.y);
    b.z = sum_rowgroups<QB>(b.z);
    b.w = sum_rowgroups<QB>(b.w);
    if (lane < QB) {
      red[buf][w][cq][0] = a;
      red[buf][w][cq][1] = b;
    }
    __syncthreads();

    a = red[buf][0][cq][0];
    b = red[buf][0][cq][1];
#pragma unroll
    for (int i = 1; i < NW; ++i) {
      const float4 ai = red[buf][i][cq][0], bi = red[buf][i][cq][1];
      a = make_float4(a.x + ai.x, a.y + ai.y, a.z + ai.z, a.w + ai.w);
      b = make_float4(b.x + bi.x, b.y + bi.y, b.z + bi.z, b.w + bi.w);
    }
    float kq = kqp[buf][0];
#pragma unroll
    for (int i = 1; i < KW; ++i) kq += kqp[buf][i];
    const float4 u = make_float4(bt * vt.x - btt * a.x, bt * vt.y - btt * a.y,
                                 bt * vt.z - btt * a.z, bt * vt.w - btt * a.w);
    if (tid < QB) {
      const float4 ov = make_float4(alpha * b.x + kq * u.x, alpha * b.y + kq * u.y,
                                    alpha * b.z + kq * u.z, alpha * b.w + kq * u.w);
      *reinterpret_cast<float4*>(o + ((long)(t0 + t) * H + h) * DV + j0 + 4 * cq) = ov;
    }
    // H <- alpha H + k u^T (k read again: holding it would cost RPT registers)
#pragma unroll
    for (int m = 0; m < RPT; m += 4) {
      const float4 k4 = *reinterpret_cast<const float4*>(&Ks[buf][lpos + m]);
      const float kr[4] = {k4.x, k4.y, k4.z, k4.w};
#pragma unroll
      for (int e = 0; e < 4; ++e)
        hs[m + e] = make_float4(fmaf(alpha, hs[m + e].x, kr[e] * u.x),
                                fmaf(alpha, hs[m + e].y, kr[e] * u.y),
                                fmaf(alpha, hs[m + e].z, kr[e] * u.z),
                                fmaf(alpha, hs[m + e].w, kr[e] * u.w));
    }
  }
  if (ht) {
#pragma unroll
    for (int m = 0; m < RPT; ++m)
      store4_stream(ht + soff + (long)RGW * m * DV, hs[m]);
  }
}

template <typename Tin, int DK, int DV, int BV, int NW>
static hipError_t launch_rec(const RecurrentArgs& a) {
  k_recurrent<Tin, DK, DV, BV, NW><<<dim3(a.N, a.H, DV / BV), 64 * NW, 0, a.stream>>>(
      static_cast<const Tin*>(a.q), static_cast<const Tin*>(a.k), static_cast<const Tin*>(a.v),
      a.g, static_cast<const Tin*>(a.beta), static_cast<const Tin*>(a.beta_tilde), a.d,
      a.cu_seqlens, a.Tseq, a.Ttot, a.H, a.h0, a.o, a.ht);
  return hipGetLastError();
}

template <typename Tin, int DK, int DV>
static hipError_t run_recurrent(const RecurrentArgs& a) {
  // at most 128 columns per workgroup and 32 rows per wave: 64 state
  // registers per lane (a d = 256 state takes two workgroups of 8 waves)
  constexpr int BV = DV < 128 ? DV : 128, NW = DK <= 128 ? 4 : DK / 32;
  a.stage("recurrent");
  hipError_t e;
  if ((long)a.N * a.H * (DV / BV) < 1024)
    // few states (small decoding batches): 32-column slices give four times
    // the workgroups, so more CUs stream the states
    e = launch_rec<Tin, DK, DV, 32, DK / 32>(a);  // 32 rows per wave: 4 per lane
  else
    e = launch_rec<Tin, DK, DV, BV, NW>(a);
  a.stage(nullptr);
  return e;
}

template <typename Tin>
static hipError_t run_recurrent_t(const RecurrentArgs& a) {
  if (a.dk == 64 && a.dv == 64) return run_recurrent<Tin, 64, 64>(a);
  if (a.dk == 64 && a.dv == 128) return run_recurrent<Tin, 64, 128>(a);
  if (a.dk == 128 && a.dv == 64) return run_recurrent<Tin, 128, 64>(a);
  if (a.dk == 128 && a.dv == 128) return run_recurrent<Tin, 128, 128>(a);
  if (a.dk == 256 && a.dv == 256) return run_recurrent<Tin, 256, 256>(a);
  if (a.dk == 128 && a.dv == 256) return run_recurrent<Tin, 128, 256>(a);
  if (a.dk == 256 && a.dv == 128) return run_recurrent<Tin, 256, 128>(a);
  return hipErrorInvalidValue;
}

hipError_t launch_recurrent(const RecurrentArgs& a) {
  if (a.N == 0) return hipSuccess;
  return a.bf16 ? run_recurrent_t<bf16_t>(a) : run_recurrent_t<float>(a);
}

}  // namespace comba
