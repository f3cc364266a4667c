// Chunk-wise Comba forward and backward for gfx950 (MI355X).
//
// Notation (per sequence, head and chunk of C = 64 tokens, rows r = 0..63):
//   G_r   in-chunk cumulative log-gate sum_{j<=r} g_j; Gm_r = G_{r-1} (Gm_0 = 0)
//   X     state entering the chunk, H = S^T in R^{dk x dv} (the paper's S_[t])
//   L     strictly lower, L_ri = beta_r exp(Gm_r - G_i) k_r.k_i       (Eq. prepare-WY_M)
//   M     (I + L)^{-1}, by forward substitution in fp32           (Section 3.3)
//   A     (Q - d K) K^T masked to r >= i and scaled by exp(G_r - G_i)
//   R     Diag(beta) V - Diag(beta exp(Gm)) K X
//   D     M R = U - W X, the pseudo-value term of the matrix form
//   O     Diag(exp G) (Q - d K) X + A D
//   X'    exp(G_63) X + K^T Diag(exp(G_63 - G_r)) D
// (W = M Diag(beta exp(Gm)) K and U = M Diag(beta) V of the paper are never
// formed: W X is evaluated as M (Diag(s) K X), which keeps every large product on
// an exact bf16 operand.)  Rows past a sequence's end are zero-filled (k = q =
// v = beta = g = 0), which makes them inert in every product.
//
// Backward (reverse mode of the same chunk form; Y = dL/dX' for the chunk):
//   dD  = A^T dO + Diag(exp(G_63 - G)) K Y,   dR = M^T dD
//   dX  = exp(G_63) Y + Q^T Diag(exp G) dO + K^T (-d Diag(exp G) dO - Diag(s) dR)
//   dL  = -strictlower(dR D^T)   (from dM = dD R^T and d(M) = -M d(L) M)
//   dA  = tril(dO D^T) ...       (the intra-chunk kernel collects the rest)
//
// Kernels, in launch order:
//   k_chunk_map  sequence/chunk tables from cu_seqlens (fixed-length rows too)
//   k_prep       per chunk-head: G, A, M                        (chunk-parallel)
//   k_scan_fwd   per (sequence, head, 32-column slice of dv): the sequential
//                state recurrence over chunks, fused with the output
//   k_scan_bwd   the reverse recurrence of the state gradient
//   k_intra_bwd  per chunk-head gradients dq, dk, dv, dbeta, dg, partial dd
//   k_reduce_dd  deterministic sum of the partial dd over chunks
#include <hip/hip_runtime.h>

#include "comba_device.hpp"
#include "comba_launch.h"

namespace comba {

// ---------------------------------------------------------------------------
// sequence / chunk tables
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(NTHR) void k_chunk_map(const int32_t* __restrict__ cu, int N, int Tseq,
                                                    int Ttot, int ncmax, ChunkInfo* __restrict__ cmap,
                                                    SeqInfo* __restrict__ smap) {
  __shared__ int wave_tot[NWAVE];
  __shared__ int carry;
  const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
  if (tid == 0) carry = 0;
  __syncthreads();
  for (int base = 0; base < N; base += NTHR) {
    const int s = base + tid;
    int tok0 = 0, len = 0, nck = 0;
    if (s < N) {
      if (cu) {
        // clamp into [0, Ttot] so that malformed offsets cannot address memory
        // outside the token range
        int a = cu[s], b = cu[s + 1];
        a = min(max(a, 0), Ttot);
        b = min(max(b, a), Ttot);
        tok0 = a;
        len = b - a;
      } else {
        tok0 = s * Tseq;
        len = Tseq;
      }
      nck = (len + CH - 1) / CH;
    }
    // exclusive scan of nck over the workgroup
    int x = nck;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int y = __shfl_up(x, off);
      if (lane >= off) x += y;
    }
    if (lane == 63) wave_tot[w] = x;
    __syncthreads();
    int before = carry;
    for (int i = 0; i < w; ++i) before += wave_tot[i];
    const int chunk0 = before + x - nck;
    if (s < N) {
      const int room = max(0, ncmax - chunk0);
      const int n = min(nck, room);
      SeqInfo si;
      si.chunk0 = chunk0;
      si.nchunks = n;
      si.tok0 = tok0;
      si.len = len;
      smap[s] = si;
      for (int j = 0; j < n; ++j) {
        ChunkInfo ci;
        ci.tok0 = tok0 + j * CH;
        ci.len = min(CH, len - j * CH);
        ci.seq = s;
        ci.pad = 0;
        cmap[chunk0 + j] = ci;
      }
    }
    __syncthreads();
    if (tid == 0) {
      int t = carry;
      for (int i = 0; i < NWAVE; ++i) t += wave_tot[i];
      carry = t;
    }
    __syncthreads();
  }
  const int total = min(carry, ncmax);
  for (int c = total + tid; c < ncmax; c += NTHR) {
    ChunkInfo ci;
    ci.tok0 = 0;
    ci.len = 0;
    ci.seq = -1;
    ci.pad = 0;
    cmap[c] = ci;
  }
}

// ---------------------------------------------------------------------------
// k_prep: per chunk-head, cumulative gates G, the masked score matrix A and the
// UT-transform inverse M = (I + L)^{-1} (Eq. prepare-WY_M), all fp32.
// ---------------------------------------------------------------------------
template <typename Tin, int DK>
__global__ __launch_bounds__(NTHR) void k_prep(const Tin* __restrict__ q, const Tin* __restrict__ k,
                                               const float* __restrict__ g,
                                               const Tin* __restrict__ beta,
                                               const float* __restrict__ d,
                                               const ChunkInfo* __restrict__ cmap, int H,
                                               float* __restrict__ Mw, float* __restrict__ Aw,
                                               float* __restrict__ Gw) {
  constexpr bool F32 = is_f32<Tin>::value;
  constexpr int LDK = DK + Pad<Tin>::value;
  constexpr int LDL = CH + 4;
  __shared__ __align__(16) Tin Ks[CH * LDK];
  __shared__ __align__(16) Tin Qs[CH * LDK];
  __shared__ __align__(16) float Ls[CH * LDL];
  __shared__ float Gs[CH], Bs[CH];

  const ChunkInfo ci = cmap[blockIdx.x];
  if (ci.len <= 0) return;
  const int h = blockIdx.y;
  const long chh = (long)blockIdx.x * H + h;
  const long tok = (long)ci.tok0 * H + h;
  const int w = wave_id(), lane = lane_id();

  tile_to_lds<Tin, CH, DK>(k + tok * DK, (long)H * DK, ci.len, Ks, LDK);
  tile_to_lds<Tin, CH, DK>(q + tok * DK, (long)H * DK, ci.len, Qs, LDK);
  if (w == 0) {
    const float gr = lane < ci.len ? g[tok + (long)lane * H] : 0.f;
    const float G = wave_prefix_sum(gr);
    Gs[lane] = G;
    Bs[lane] = lane < ci.len ? to_f(beta[tok + (long)lane * H]) : 0.f;
    Gw[chh * CH + lane] = G;
  }
  __syncthreads();

  // A_kk = K K^T and A_qk = Q K^T for rows 16w..16w+15
  floatx4 akk[1][4], aqk[1][4];
  zero_acc(akk);
  zero_acc(aqk);
  mma<F32, 1, 4, DK>(akk, Ks + 16 * w * LDK, LDK, Ks, LDK);
  mma<F32, 1, 4, DK>(aqk, Qs + 16 * w * LDK, LDK, Ks, LDK);
  const float dh = d[h];
#pragma unroll
  for (int nt = 0; nt < 4; ++nt)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = 16 * w + acc_row(0, e), c = acc_col(nt);
      const float kk = akk[0][nt][e];
      float a = 0.f, l = 0.f;
      if (r >= c) a = (aqk[0][nt][e] - dh * kk) * __expf(Gs[r] - Gs[c]);
      if (r > c) {
        const float gm = Gs[r - 1];
        l = Bs[r] * __expf(gm - Gs[c]) * kk;
      }
      Aw[chh * CH * CH + r * CH + c] = a;
      Ls[r * LDL + c] = l;
    }
  __syncthreads();

  // M = (I + L)^{-1}: lane j solves column j by forward substitution,
  // x_i = -sum_{j <= m < i} L_im x_m, with x_j = 1 (rows processed in order).
  if (w == 0) {
    const int j = lane;
    float x[CH];
#pragma unroll
    for (int i = 0; i < CH; ++i) x[i] = (i == j) ? 1.f : 0.f;
#pragma unroll
    for (int i = 1; i < CH; ++i) {
      float s = 0.f;
#pragma unroll
      for (int m = 0; m < i; m += 4) {
        const float4 lv = *reinterpret_cast<const float4*>(Ls + i * LDL + m);
        s += lv.x * x[m];
        if (m + 1 < i) s += lv.y * x[m + 1];
        if (m + 2 < i) s += lv.z * x[m + 2];
        if (m + 3 < i) s += lv.w * x[m + 3];
      }
      if (i > j) x[i] = -s;
    }
    float* Mo = Mw + chh * CH * CH;
#pragma unroll
    for (int i = 0; i < CH; ++i) Mo[i * CH + j] = x[i];
  }
}

// ---------------------------------------------------------------------------
// k_scan_fwd: one workgroup per (sequence, head, 32-wide dv slice) walks the
// chunks of its sequence in order, keeping its dk x 32 state slice in fp32.
//   OUT   : write the outputs o (forward entry point)
//   STORE : save the entering state X and D per chunk (backward recompute)
// ---------------------------------------------------------------------------
template <typename Tin, int DK, int DV, bool OUT, bool STORE>
__global__ __launch_bounds__(NTHR, 1) void k_scan_fwd(
    const Tin* __restrict__ q, const Tin* __restrict__ k, const Tin* __restrict__ v,
    const Tin* __restrict__ beta, const float* __restrict__ d, const float* __restrict__ h0,
    const ChunkInfo* __restrict__ cmap, const SeqInfo* __restrict__ smap, int H,
    const float* __restrict__ Mw, const float* __restrict__ Aw, const float* __restrict__ Gw,
    float* __restrict__ o, float* __restrict__ ht, float* __restrict__ Xw, float* __restrict__ Dw) {
  constexpr bool F32 = is_f32<Tin>::value;
  constexpr int BV = 32, NTV = BV / 16, XMT = DK / 64;
  constexpr int PI = Pad<Tin>::value;
  constexpr int LDK = DK + PI, LDC = CH + PI, LDV = BV + PI;
  constexpr int LDF = CH + 4, LDX = DK + 4;
  __shared__ __align__(16) Tin Ks[CH * LDK];
  __shared__ __align__(16) Tin KsT[DK * LDC];
  __shared__ __align__(16) Tin Qs[OUT ? CH * LDK : 8];
  __shared__ __align__(16) Tin Vs[CH * LDV];
  __shared__ __align__(16) float Ms[CH * LDF];
  __shared__ __align__(16) float As[OUT ? CH * LDF : 4];
  __shared__ __align__(16) float XT[BV * LDX];
  __shared__ __align__(16) float RT[BV * LDF];
  __shared__ __align__(16) float DT[OUT ? BV * LDF : 4];
  __shared__ __align__(16) float DgT[BV * LDF];
  __shared__ float Gs[CH], Bs[CH];

  const int s = blockIdx.x, h = blockIdx.y, j0 = blockIdx.z * BV;
  const SeqInfo si = smap[s];
  const int w = wave_id();
  const long soff = ((long)s * H + h) * DK * DV;
  const float dh = d[h];

  floatx4 X[XMT][NTV];
#pragma unroll
  for (int mt = 0; mt < XMT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NTV; ++nt)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int i = (DK / 4) * w + acc_row(mt, e), jj = acc_col(nt);
        X[mt][nt][e] = h0 ? h0[soff + (long)i * DV + j0 + jj] : 0.f;
        XT[jj * LDX + i] = X[mt][nt][e];
      }

  for (int cc = 0; cc < si.nchunks; ++cc) {
    const int c = si.chunk0 + cc;
    const ChunkInfo ci = cmap[c];
    const long chh = (long)c * H + h;
    const long tok = (long)ci.tok0 * H + h;
    __syncthreads();
    tile_to_lds_t<Tin, CH, DK, true>(k + tok * DK, (long)H * DK, ci.len, Ks, LDK, KsT, LDC);
    if constexpr (OUT) tile_to_lds<Tin, CH, DK>(q + tok * DK, (long)H * DK, ci.len, Qs, LDK);
    tile_to_lds<Tin, CH, BV>(v + tok * DV + j0, (long)H * DV, ci.len, Vs, LDV);
    tile_to_lds<float, CH, CH>(Mw + chh * CH * CH, CH, CH, Ms, LDF);
    if constexpr (OUT) tile_to_lds<float, CH, CH>(Aw + chh * CH * CH, CH, CH, As, LDF);
    if (threadIdx.x < CH) {
      const int r = threadIdx.x;
      Gs[r] = Gw[chh * CH + r];
      Bs[r] = r < ci.len ? to_f(beta[tok + (long)r * H]) : 0.f;
    }
    if constexpr (STORE) {
#pragma unroll
      for (int mt = 0; mt < XMT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NTV; ++nt)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int i = (DK / 4) * w + acc_row(mt, e), jj = acc_col(nt);
            Xw[chh * DK * DV + (long)i * DV + j0 + jj] = X[mt][nt][e];
          }
    }
    __syncthreads();
    const float Glast = Gs[CH - 1];

    // K X and Q X for rows 16w..16w+15; R = Diag(beta)(V - Diag(exp Gm) K X)
    floatx4 kx[1][NTV], qx[1][NTV];
    zero_acc(kx);
    mma<F32, 1, NTV, DK>(kx, Ks + 16 * w * LDK, LDK, XT, LDX);
    if constexpr (OUT) {
      zero_acc(qx);
      mma<F32, 1, NTV, DK>(qx, Qs + 16 * w * LDK, LDK, XT, LDX);
    }
    floatx4 oacc[1][NTV];
#pragma unroll
    for (int nt = 0; nt < NTV; ++nt)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 16 * w + acc_row(0, e), jj = acc_col(nt);
        const float kxv = kx[0][nt][e];
        const float gm = r > 0 ? Gs[r - 1] : 0.f;
        RT[jj * LDF + r] = Bs[r] * (to_f(Vs[r * LDV + jj]) - __expf(gm) * kxv);
        if constexpr (OUT) oacc[0][nt][e] = __expf(Gs[r]) * (qx[0][nt][e] - dh * kxv);
      }
    __syncthreads();

    // D = M R
    floatx4 dl[1][NTV];
    zero_acc(dl);
    mma<F32, 1, NTV, CH>(dl, Ms + 16 * w * LDF, LDF, RT, LDF);
#pragma unroll
    for (int nt = 0; nt < NTV; ++nt)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 16 * w + acc_row(0, e), jj = acc_col(nt);
        const float dv = dl[0][nt][e];
        if constexpr (OUT) DT[jj * LDF + r] = dv;
        DgT[jj * LDF + r] = __expf(Glast - Gs[r]) * dv;
        if constexpr (STORE) Dw[chh * CH * DV + (long)r * DV + j0 + jj] = dv;
      }
    __syncthreads();

    // X' = exp(G_63) X + K^T Diag(exp(G_63 - G)) D
    const float gC = __expf(Glast);
#pragma unroll
    for (int mt = 0; mt < XMT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt) X[mt][nt] *= gC;
    mma<F32, XMT, NTV, CH>(X, KsT + (DK / 4) * w * LDC, LDC, DgT, LDF);

    // O = Diag(exp G)(Q - d K) X + A D
    if constexpr (OUT) {
      mma<F32, 1, NTV, CH>(oacc, As + 16 * w * LDF, LDF, DT, LDF);
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = 16 * w + acc_row(0, e), jj = acc_col(nt);
          if (r < ci.len) o[(tok + (long)r * H) * DV + j0 + jj] = oacc[0][nt][e];
        }
    }
#pragma unroll
    for (int mt = 0; mt < XMT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          XT[acc_col(nt) * LDX + (DK / 4) * w + acc_row(mt, e)] = X[mt][nt][e];
  }
  if (ht) {
#pragma unroll
    for (int mt = 0; mt < XMT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int i = (DK / 4) * w + acc_row(mt, e), jj = acc_col(nt);
          ht[soff + (long)i * DV + j0 + jj] = X[mt][nt][e];
        }
  }
}

// ---------------------------------------------------------------------------
// k_scan_bwd: reverse recurrence of Y = dL/d(state leaving the chunk).
// Saves Y (as seen by each chunk) and dR = M^T dD per chunk for k_intra_bwd.
// ---------------------------------------------------------------------------
template <typename Tin, int DK, int DV>
__global__ __launch_bounds__(NTHR, 1) void k_scan_bwd(
    const Tin* __restrict__ q, const Tin* __restrict__ k, const Tin* __restrict__ dO,
    const Tin* __restrict__ beta, const float* __restrict__ d, const float* __restrict__ dht,
    const ChunkInfo* __restrict__ cmap, const SeqInfo* __restrict__ smap, int H,
    const float* __restrict__ Mw, const float* __restrict__ Aw, const float* __restrict__ Gw,
    float* __restrict__ dh0, float* __restrict__ Yw, float* __restrict__ dRw) {
  constexpr bool F32 = is_f32<Tin>::value;
  constexpr int BV = 32, NTV = BV / 16, XMT = DK / 64;
  constexpr int PI = Pad<Tin>::value;
  constexpr int LDK = DK + PI, LDC = CH + PI;
  constexpr int LDF = CH + 4, LDX = DK + 4;
  __shared__ __align__(16) Tin Ks[CH * LDK];
  __shared__ __align__(16) Tin KsT[DK * LDC];
  __shared__ __align__(16) Tin QsT[DK * LDC];
  __shared__ __align__(16) Tin dOT[BV * LDC];
  __shared__ __align__(16) float AsT[CH * LDF];
  __shared__ __align__(16) float MsT[CH * LDF];
  __shared__ __align__(16) float YT[BV * LDX];
  __shared__ __align__(16) float dDT[BV * LDF];
  __shared__ __align__(16) float PgT[BV * LDF];
  __shared__ __align__(16) float W2T[BV * LDF];
  __shared__ float Gs[CH], Bs[CH];

  const int s = blockIdx.x, h = blockIdx.y, j0 = blockIdx.z * BV;
  const SeqInfo si = smap[s];
  const int w = wave_id();
  const long soff = ((long)s * H + h) * DK * DV;
  const float dh = d[h];

  floatx4 Y[XMT][NTV];
#pragma unroll
  for (int mt = 0; mt < XMT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NTV; ++nt)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int i = (DK / 4) * w + acc_row(mt, e), jj = acc_col(nt);
        Y[mt][nt][e] = dht ? dht[soff + (long)i * DV + j0 + jj] : 0.f;
        YT[jj * LDX + i] = Y[mt][nt][e];
      }

  for (int cc = si.nchunks - 1; cc >= 0; --cc) {
    const int c = si.chunk0 + cc;
    const ChunkInfo ci = cmap[c];
    const long chh = (long)c * H + h;
    const long tok = (long)ci.tok0 * H + h;
    __syncthreads();
    tile_to_lds_t<Tin, CH, DK, true>(k + tok * DK, (long)H * DK, ci.len, Ks, LDK, KsT, LDC);
    tile_to_lds_t<Tin, CH, DK, false>(q + tok * DK, (long)H * DK, ci.len, nullptr, 0, QsT, LDC);
    tile_to_lds_t<Tin, CH, BV, false>(dO + tok * DV + j0, (long)H * DV, ci.len, nullptr, 0, dOT, LDC);
    tile_to_lds_t<float, CH, CH, false>(Aw + chh * CH * CH, CH, CH, nullptr, 0, AsT, LDF);
    tile_to_lds_t<float, CH, CH, false>(Mw + chh * CH * CH, CH, CH, nullptr, 0, MsT, LDF);
    if (threadIdx.x < CH) {
      const int r = threadIdx.x;
      Gs[r] = Gw[chh * CH + r];
      Bs[r] = r < ci.len ? to_f(beta[tok + (long)r * H]) : 0.f;
    }
#pragma unroll
    for (int mt = 0; mt < XMT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int i = (DK / 4) * w + acc_row(mt, e), jj = acc_col(nt);
          Yw[chh * DK * DV + (long)i * DV + j0 + jj] = Y[mt][nt][e];
        }
    __syncthreads();
    const float Glast = Gs[CH - 1];

    // dD = A^T dO + Diag(exp(G_63 - G)) K Y
    floatx4 ky[1][NTV], ad[1][NTV];
    zero_acc(ky);
    zero_acc(ad);
    mma<F32, 1, NTV, DK>(ky, Ks + 16 * w * LDK, LDK, YT, LDX);
    mma<F32, 1, NTV, CH>(ad, AsT + 16 * w * LDF, LDF, dOT, LDC);
#pragma unroll
    for (int nt = 0; nt < NTV; ++nt)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 16 * w + acc_row(0, e), jj = acc_col(nt);
        dDT[jj * LDF + r] = ad[0][nt][e] + __expf(Glast - Gs[r]) * ky[0][nt][e];
      }
    __syncthreads();

    // dR = M^T dD;  Pg = Diag(exp G) dO;  W2 = -d Pg - Diag(beta exp Gm) dR
    floatx4 dr[1][NTV];
    zero_acc(dr);
    mma<F32, 1, NTV, CH>(dr, MsT + 16 * w * LDF, LDF, dDT, LDF);
#pragma unroll
    for (int nt = 0; nt < NTV; ++nt)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 16 * w + acc_row(0, e), jj = acc_col(nt);
        const float drv = dr[0][nt][e];
        dRw[chh * CH * DV + (long)r * DV + j0 + jj] = drv;
        const float pg = __expf(Gs[r]) * to_f(dOT[jj * LDC + r]);
        const float gm = r > 0 ? Gs[r - 1] : 0.f;
        PgT[jj * LDF + r] = pg;
        W2T[jj * LDF + r] = -dh * pg - Bs[r] * __expf(gm) * drv;
      }
    __syncthreads();

    // Y <- exp(G_63) Y + Q^T Pg + K^T W2
    const float gC = __expf(Glast);
#pragma unroll
    for (int mt = 0; mt < XMT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt) Y[mt][nt] *= gC;
    mma<F32, XMT, NTV, CH>(Y, QsT + (DK / 4) * w * LDC, LDC, PgT, LDF);
    mma<F32, XMT, NTV, CH>(Y, KsT + (DK / 4) * w * LDC, LDC, W2T, LDF);
#pragma unroll
    for (int mt = 0; mt < XMT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          YT[acc_col(nt) * LDX + (DK / 4) * w + acc_row(mt, e)] = Y[mt][nt][e];
  }
  if (dh0) {
#pragma unroll
    for (int mt = 0; mt < XMT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int i = (DK / 4) * w + acc_row(mt, e), jj = acc_col(nt);
          dh0[soff + (long)i * DV + j0 + jj] = Y[mt][nt][e];
        }
  }
}

// ---------------------------------------------------------------------------
// k_intra_bwd: per chunk-head gradients.  Phase 1 streams the dv axis in blocks
// of 32 and accumulates the dv-reductions
//   T1 = dO X^T, T3 = dR X^T, T2 = D Y^T (C x dk), dO D^T, dR D^T (C x C),
//   <Y, X>_F, <v_r, dR_r>, and writes dv = Diag(beta) dR.
// Phase 2 forms
//   dQ~ = Diag(exp G) T1 + (dA o Gamma) K
//   dK  = Diag(exp(G_63 - G)) T2 - Diag(s) T3 + (dA o Gamma)^T Q
//         + (dAkk + dAkk^T - d (dA o Gamma)^T) K
// and the per-token gate / beta gradients, then dg by a reverse in-chunk sum.
// ---------------------------------------------------------------------------
template <typename Tin, int DK, int DV>
struct IntraBwdSmem {
  static constexpr int VB = 32;
  static constexpr int PI = Pad<Tin>::value;
  static constexpr int LDK = DK + PI, LDC = CH + PI, LDVB = VB + PI;
  static constexpr int LDF = CH + 4, LDFB = VB + 4;
  static constexpr int P1 = 2 * CH * LDVB * (int)sizeof(Tin) + 2 * CH * LDFB * 4 + 2 * DK * LDFB * 4;
  static constexpr int P2 = 2 * CH * LDK * (int)sizeof(Tin) + 2 * DK * LDC * (int)sizeof(Tin) +
                            4 * CH * LDF * 4;
  static constexpr int BYTES = P1 > P2 ? P1 : P2;
};

template <typename Tin, int DK, int DV>
__global__ __launch_bounds__(NTHR, 1) void k_intra_bwd(
    const Tin* __restrict__ q, const Tin* __restrict__ k, const Tin* __restrict__ v,
    const Tin* __restrict__ dO, const Tin* __restrict__ beta, const float* __restrict__ d,
    const ChunkInfo* __restrict__ cmap, int H, const float* __restrict__ Gw,
    const float* __restrict__ Xw, const float* __restrict__ Dw, const float* __restrict__ Yw,
    const float* __restrict__ dRw, float* __restrict__ dq, float* __restrict__ dk,
    float* __restrict__ dv, float* __restrict__ dbeta, float* __restrict__ dg,
    float* __restrict__ ddp) {
  using SM = IntraBwdSmem<Tin, DK, DV>;
  constexpr bool F32 = is_f32<Tin>::value;
  constexpr int VB = SM::VB, LDK = SM::LDK, LDC = SM::LDC, LDVB = SM::LDVB, LDF = SM::LDF,
                LDFB = SM::LDFB;
  constexpr int NTK = DK / 16;
  __shared__ __align__(16) char smem[SM::BYTES];
  __shared__ float Gs[CH], Bs[CH], rowG[CH], rowGm[CH], rowB[CH];
  __shared__ float colpart[NWAVE][CH];
  __shared__ float scal[NWAVE][3];

  const int h = blockIdx.y;
  const long chh = (long)blockIdx.x * H + h;
  const ChunkInfo ci = cmap[blockIdx.x];
  if (ci.len <= 0) {
    if (threadIdx.x == 0) ddp[chh] = 0.f;
    return;
  }
  const long tok = (long)ci.tok0 * H + h;
  const int tid = threadIdx.x, w = wave_id(), lane = lane_id();
  const int len = ci.len;
  const float dh = d[h];

  if (tid < CH) {
    Gs[tid] = Gw[chh * CH + tid];
    Bs[tid] = tid < len ? to_f(beta[tok + (long)tid * H]) : 0.f;
    rowG[tid] = 0.f;
    rowGm[tid] = 0.f;
  }

  // ---------------- phase 1: reductions over dv ----------------
  Tin* dOb = reinterpret_cast<Tin*>(smem);
  Tin* Vb = dOb + CH * LDVB;
  float* dRb = reinterpret_cast<float*>(Vb + CH * LDVB);
  float* Dlb = dRb + CH * LDFB;
  float* Xb = Dlb + CH * LDFB;
  float* Yb = Xb + DK * LDFB;

  floatx4 T1[1][NTK], T2[1][NTK], T3[1][NTK], dAr[1][4], dLr[1][4];
  zero_acc(T1);
  zero_acc(T2);
  zero_acc(T3);
  zero_acc(dAr);
  zero_acc(dLr);
  float Fpart = 0.f, bv = 0.f;
  const int er = tid >> 2, ec = (tid & 3) * 8;  // elementwise ownership: row er, 8 columns
  for (int vb = 0; vb < DV / VB; ++vb) {
    __syncthreads();
    tile_to_lds<Tin, CH, VB>(dO + tok * DV + vb * VB, (long)H * DV, len, dOb, LDVB);
    tile_to_lds<Tin, CH, VB>(v + tok * DV + vb * VB, (long)H * DV, len, Vb, LDVB);
    tile_to_lds<float, CH, VB>(dRw + chh * CH * DV + vb * VB, DV, CH, dRb, LDFB);
    tile_to_lds<float, CH, VB>(Dw + chh * CH * DV + vb * VB, DV, CH, Dlb, LDFB);
    tile_to_lds<float, DK, VB>(Xw + chh * DK * DV + vb * VB, DV, DK, Xb, LDFB);
    tile_to_lds<float, DK, VB>(Yw + chh * DK * DV + vb * VB, DV, DK, Yb, LDFB);
    __syncthreads();
    mma<F32, 1, NTK, VB>(T1, dOb + 16 * w * LDVB, LDVB, Xb, LDFB);
    mma<F32, 1, NTK, VB>(T3, dRb + 16 * w * LDFB, LDFB, Xb, LDFB);
    mma<F32, 1, NTK, VB>(T2, Dlb + 16 * w * LDFB, LDFB, Yb, LDFB);
    mma<F32, 1, 4, VB>(dAr, dOb + 16 * w * LDVB, LDVB, Dlb, LDFB);
    mma<F32, 1, 4, VB>(dLr, dRb + 16 * w * LDFB, LDFB, Dlb, LDFB);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float x = dRb[er * LDFB + ec + e];
      bv += to_f(Vb[er * LDVB + ec + e]) * x;
      if (er < len) dv[(tok + (long)er * H) * DV + vb * VB + ec + e] = Bs[er] * x;
    }
    for (int idx = tid; idx < DK * VB; idx += NTHR) {
      const int i = idx / VB, jj = idx % VB;
      Fpart += Xb[i * LDFB + jj] * Yb[i * LDFB + jj];
    }
  }
  bv += __shfl_xor(bv, 1);
  bv += __shfl_xor(bv, 2);
  if ((tid & 3) == 0) rowB[er] = bv;
  Fpart = wave_sum(Fpart);
  if (lane == 0) scal[w][0] = Fpart;
  __syncthreads();

  // ---------------- phase 2 ----------------
  Tin* Ks = reinterpret_cast<Tin*>(smem);
  Tin* Qs = Ks + CH * LDK;
  Tin* KsT = Qs + CH * LDK;
  Tin* QsT = KsT + DK * LDC;
  float* dAG = reinterpret_cast<float*>(QsT + DK * LDC);
  float* dAGT = dAG + CH * LDF;
  float* Bsym = dAGT + CH * LDF;
  float* dAkk = Bsym + CH * LDF;
  tile_to_lds_t<Tin, CH, DK, true>(k + tok * DK, (long)H * DK, len, Ks, LDK, KsT, LDC);
  tile_to_lds_t<Tin, CH, DK, true>(q + tok * DK, (long)H * DK, len, Qs, LDK, QsT, LDC);
  __syncthreads();
  const float Glast = Gs[CH - 1];

  {
    floatx4 akk[1][4], aqk[1][4];
    zero_acc(akk);
    zero_acc(aqk);
    mma<F32, 1, 4, DK>(akk, Ks + 16 * w * LDK, LDK, Ks, LDK);
    mma<F32, 1, 4, DK>(aqk, Qs + 16 * w * LDK, LDK, Ks, LDK);
    float rE1[4] = {0.f, 0.f, 0.f, 0.f}, rE2[4] = {0.f, 0.f, 0.f, 0.f}, rBL[4] = {0.f, 0.f, 0.f, 0.f};
    float cE[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 16 * w + acc_row(0, e), c = acc_col(nt);
        const float kk = akk[0][nt][e];
        float dag = 0.f, e1 = 0.f, e2 = 0.f, dakk = 0.f;
        if (r >= c) {
          const float gam = __expf(Gs[r] - Gs[c]);
          const float a = (aqk[0][nt][e] - dh * kk) * gam;
          const float da = dAr[0][nt][e];
          e1 = da * a;
          dag = da * gam;
        }
        if (r > c) {
          const float lc = __expf(Gs[r - 1] - Gs[c]);
          const float dl = -dLr[0][nt][e];
          const float lck = lc * kk;
          e2 = dl * Bs[r] * lck;
          rBL[e] += dl * lck;
          dakk = dl * Bs[r] * lc;
        }
        rE1[e] += e1;
        rE2[e] += e2;
        cE[nt] += e1 + e2;
        dAG[r * LDF + c] = dag;
        dAGT[c * LDF + r] = dag;
        dAkk[r * LDF + c] = dakk;
      }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      rE1[e] = sum16(rE1[e]);
      rE2[e] = sum16(rE2[e]);
      rBL[e] = sum16(rBL[e]);
    }
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      cE[nt] = sum_groups(cE[nt]);
      if ((lane >> 4) == 0) colpart[w][acc_col(nt)] = cE[nt];
    }
    if ((lane & 15) == 0) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 16 * w + acc_row(0, e);
        rowG[r] += rE1[e];
        rowGm[r] += rE2[e];
        rowB[r] += rBL[e];
      }
    }
  }
  __syncthreads();
  for (int idx = tid; idx < CH * CH; idx += NTHR) {
    const int r = idx / CH, c = idx % CH;
    Bsym[r * LDF + c] = dAkk[r * LDF + c] + dAkk[c * LDF + r] - dh * dAGT[r * LDF + c];
  }
  __syncthreads();

  // row dot products of T1, T2, T3 with q~ and k
  {
    float p1[4] = {0.f, 0.f, 0.f, 0.f}, p2[4] = {0.f, 0.f, 0.f, 0.f}, p3[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int nt = 0; nt < NTK; ++nt)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 16 * w + acc_row(0, e), c = acc_col(nt);
        const float kv = to_f(Ks[r * LDK + c]);
        const float qv = to_f(Qs[r * LDK + c]) - dh * kv;
        p1[e] += T1[0][nt][e] * qv;
        p2[e] += T2[0][nt][e] * kv;
        p3[e] += T3[0][nt][e] * kv;
      }
    float gcp = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      p1[e] = sum16(p1[e]);
      p2[e] = sum16(p2[e]);
      p3[e] = sum16(p3[e]);
      if ((lane & 15) == 0) {
        const int r = 16 * w + acc_row(0, e);
        const float cr = __expf(Glast - Gs[r]) * p2[e];
        const float egm = __expf(r > 0 ? Gs[r - 1] : 0.f);
        rowG[r] += __expf(Gs[r]) * p1[e] - cr;
        rowGm[r] -= Bs[r] * egm * p3[e];
        rowB[r] -= egm * p3[e];
        gcp += cr;
      }
    }
    gcp = wave_sum(gcp);
    if (lane == 0) scal[w][1] = gcp;
  }

  // dQ~ (in T1) and dK (in T2)
#pragma unroll
  for (int nt = 0; nt < NTK; ++nt)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = 16 * w + acc_row(0, e);
      const float egm = __expf(r > 0 ? Gs[r - 1] : 0.f);
      T1[0][nt][e] *= __expf(Gs[r]);
      T2[0][nt][e] = __expf(Glast - Gs[r]) * T2[0][nt][e] - Bs[r] * egm * T3[0][nt][e];
    }
  mma<F32, 1, NTK, CH>(T1, dAG + 16 * w * LDF, LDF, KsT, LDC);
  mma<F32, 1, NTK, CH>(T2, dAGT + 16 * w * LDF, LDF, QsT, LDC);
  mma<F32, 1, NTK, CH>(T2, Bsym + 16 * w * LDF, LDF, KsT, LDC);
  float ddpart = 0.f;
#pragma unroll
  for (int nt = 0; nt < NTK; ++nt)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = 16 * w + acc_row(0, e), c = acc_col(nt);
      const float dqt = T1[0][nt][e];
      ddpart += to_f(Ks[r * LDK + c]) * dqt;
      if (r < len) {
        const long off = (tok + (long)r * H) * DK + c;
        dq[off] = dqt;
        dk[off] = T2[0][nt][e] - dh * dqt;
      }
    }
  ddpart = wave_sum(ddpart);
  if (lane == 0) scal[w][2] = ddpart;
  __syncthreads();

  if (w == 0) {
    const int r = lane;
    float F = 0.f, gcs = 0.f, dds = 0.f, col = 0.f;
#pragma unroll
    for (int i = 0; i < NWAVE; ++i) {
      F += scal[i][0];
      gcs += scal[i][1];
      dds += scal[i][2];
      col += colpart[i][r];
    }
    float dG = rowG[r] - col + (r + 1 < CH ? rowGm[r + 1] : 0.f);
    if (r == CH - 1) dG += gcs + __expf(Glast) * F;
    // dg_r = sum_{r' >= r} dG_r' (reverse in-chunk cumulative sum)
    float x = __shfl(dG, 63 - lane);
    x = wave_prefix_sum(x);
    const float dgr = __shfl(x, 63 - lane);
    if (r < len) {
      dg[tok + (long)r * H] = dgr;
      dbeta[tok + (long)r * H] = rowB[r];
    }
    if (lane == 0) ddp[chh] = -dds;
  }
}

// dd[h] = sum over chunks of the per-chunk partials (fixed order)
__global__ __launch_bounds__(NTHR) void k_reduce_dd(const float* __restrict__ ddp, int nc, int H,
                                                    float* __restrict__ dd) {
  __shared__ float part[NTHR];
  const int h = blockIdx.x;
  float s = 0.f;
  for (int c = threadIdx.x; c < nc; c += NTHR) s += ddp[(long)c * H + h];
  part[threadIdx.x] = s;
  __syncthreads();
  for (int off = NTHR / 2; off > 0; off >>= 1) {
    if ((int)threadIdx.x < off) part[threadIdx.x] += part[threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x == 0) dd[h] = part[0];
}

// ---------------------------------------------------------------------------
// host launchers
// ---------------------------------------------------------------------------
template <typename Tin, int DK, int DV>
static hipError_t run_fwd(const LaunchArgs& a) {
  hipStream_t st = a.stream;
  const Tin* q = static_cast<const Tin*>(a.q);
  const Tin* k = static_cast<const Tin*>(a.k);
  const Tin* v = static_cast<const Tin*>(a.v);
  const Tin* beta = static_cast<const Tin*>(a.beta);
  a.stage("chunk_map");
  k_chunk_map<<<1, NTHR, 0, st>>>(a.cu_seqlens, a.N, a.Tseq, a.Ttot, a.ncmax, a.cmap, a.smap);
  a.stage("prep");
  if (a.ncmax > 0)
    k_prep<Tin, DK><<<dim3(a.ncmax, a.H), NTHR, 0, st>>>(q, k, a.g, beta, a.d, a.cmap, a.H, a.Mw,
                                                         a.Aw, a.Gw);
  a.stage("scan_fwd");
  k_scan_fwd<Tin, DK, DV, true, false><<<dim3(a.N, a.H, DV / 32), NTHR, 0, st>>>(
      q, k, v, beta, a.d, a.h0, a.cmap, a.smap, a.H, a.Mw, a.Aw, a.Gw, a.o, a.ht, nullptr, nullptr);
  a.stage(nullptr);
  return hipGetLastError();
}

template <typename Tin, int DK, int DV>
static hipError_t run_bwd(const LaunchArgs& a) {
  hipStream_t st = a.stream;
  const Tin* q = static_cast<const Tin*>(a.q);
  const Tin* k = static_cast<const Tin*>(a.k);
  const Tin* v = static_cast<const Tin*>(a.v);
  const Tin* beta = static_cast<const Tin*>(a.beta);
  const Tin* dO = static_cast<const Tin*>(a.dO);
  if (a.N == 0) {
    // no sequences: dd (one value per head) is zero
    k_reduce_dd<<<a.H, NTHR, 0, st>>>(a.ddp, 0, a.H, a.dd);
    return hipGetLastError();
  }
  a.stage("chunk_map");
  k_chunk_map<<<1, NTHR, 0, st>>>(a.cu_seqlens, a.N, a.Tseq, a.Ttot, a.ncmax, a.cmap, a.smap);
  a.stage("prep");
  if (a.ncmax > 0)
    k_prep<Tin, DK><<<dim3(a.ncmax, a.H), NTHR, 0, st>>>(q, k, a.g, beta, a.d, a.cmap, a.H, a.Mw,
                                                         a.Aw, a.Gw);
  a.stage("scan_fwd_store");
  k_scan_fwd<Tin, DK, DV, false, true><<<dim3(a.N, a.H, DV / 32), NTHR, 0, st>>>(
      q, k, v, beta, a.d, a.h0, a.cmap, a.smap, a.H, a.Mw, a.Aw, a.Gw, nullptr, nullptr, a.Xw,
      a.Dw);
  a.stage("scan_bwd");
  k_scan_bwd<Tin, DK, DV><<<dim3(a.N, a.H, DV / 32), NTHR, 0, st>>>(
      q, k, dO, beta, a.d, a.dht, a.cmap, a.smap, a.H, a.Mw, a.Aw, a.Gw, a.dh0, a.Yw, a.dRw);
  a.stage("intra_bwd");
  if (a.ncmax > 0)
    k_intra_bwd<Tin, DK, DV><<<dim3(a.ncmax, a.H), NTHR, 0, st>>>(
        q, k, v, dO, beta, a.d, a.cmap, a.H, a.Gw, a.Xw, a.Dw, a.Yw, a.dRw, a.dq, a.dk_, a.dv_,
        a.dbeta, a.dg, a.ddp);
  a.stage("reduce_dd");
  k_reduce_dd<<<a.H, NTHR, 0, st>>>(a.ddp, a.ncmax, a.H, a.dd);
  a.stage(nullptr);
  return hipGetLastError();
}

template <bool BWD, typename Tin>
static hipError_t dispatch_dims(const LaunchArgs& a) {
  if (a.dk == 64 && a.dv == 64) return BWD ? run_bwd<Tin, 64, 64>(a) : run_fwd<Tin, 64, 64>(a);
  if constexpr (!is_f32<Tin>::value) {
    if (a.dk == 128 && a.dv == 128) return BWD ? run_bwd<Tin, 128, 128>(a) : run_fwd<Tin, 128, 128>(a);
    if (a.dk == 64 && a.dv == 128) return BWD ? run_bwd<Tin, 64, 128>(a) : run_fwd<Tin, 64, 128>(a);
    if (a.dk == 128 && a.dv == 64) return BWD ? run_bwd<Tin, 128, 64>(a) : run_fwd<Tin, 128, 64>(a);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_fwd(const LaunchArgs& a) {
  return a.bf16 ? dispatch_dims<false, bf16_t>(a) : dispatch_dims<false, float>(a);
}

hipError_t launch_bwd(const LaunchArgs& a) {
  return a.bf16 ? dispatch_dims<true, bf16_t>(a) : dispatch_dims<true, float>(a);
}

}  // namespace comba
