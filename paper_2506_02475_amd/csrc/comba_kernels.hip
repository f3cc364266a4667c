// Chunk-wise Comba forward and backward for gfx950 (MI355X).
//
// Notation (per sequence, head and chunk of C = 64 tokens, rows r = 0..63):
//   G_r   in-chunk cumulative log-gate sum_{j<=r} g_j; Gm_r = G_{r-1} (Gm_0 = 0)
//   X     state entering the chunk, H = S^T in R^{dk x dv} (the paper's S_[t])
//   L     strictly lower, L_ri = beta_r exp(Gm_r - G_i) k_r.k_i       (Eq. prepare-WY_M)
//   M     (I + L)^{-1} in fp32 (Section 3.3): forward substitution (fp32 path);
//         blocked, substitution in the 16x16 diagonal blocks and MFMA for the rest (bf16 path)
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
//   k_seq_map, k_chunk_fill  sequence/chunk tables from cu_seqlens (fixed-length rows too)
//   k_prep       per chunk-head: G, A, M                        (chunk-parallel)
//   k_scan_fwd   per (sequence, head, 32-column slice of dv): the sequential
//                state recurrence over chunks, fused with the output
//   k_scan_bwd   the reverse recurrence of the state gradient
//   k_intra_bwd  per chunk-head gradients dq, dk, dv, dbeta (, dbeta~), dg, partial dd
//   k_reduce_dd  deterministic sum of the partial dd over chunks
#include <hip/hip_runtime.h>

#include <mutex>

#include "comba_device.hpp"
#include "comba_launch.h"

namespace comba {

// ---------------------------------------------------------------------------
// sequence / chunk tables
// ---------------------------------------------------------------------------
// k_seq_map: one workgroup; per sequence its token range (clamped into
// [0, Ttot], so that malformed offsets cannot address memory outside the token
// range) and its first chunk (exclusive scan of the chunk counts, NTHR
// sequences per pass).
// It also writes the order in which the scans take the sequences, sorder[r] =
// the sequence of rank r: longest first (ties by index) for up to SORT_MAX
// sequences, so that the longest chains start first; identity beyond that.
constexpr int SORT_MAX = 1024;
__global__ __launch_bounds__(NTHR) void k_seq_map(const int32_t* __restrict__ cu, int N, int Tseq,
                                                  int Ttot, int ncmax, SeqInfo* __restrict__ smap,
                                                  int* __restrict__ sorder) {
  __shared__ int wave_tot[NWAVE];
  __shared__ int carry;
  __shared__ int nckS[SORT_MAX];
  const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
  if (tid == 0) carry = 0;
  __syncthreads();
  for (int base = 0; base < N; base += NTHR) {
    const int s = base + tid;
    int tok0 = 0, len = 0, nck = 0;
    if (s < N) {
      if (cu) {
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
      // a sequence never reaches past the ncmax chunk slots of the workspace
      SeqInfo si;
      si.chunk0 = min(chunk0, ncmax);
      si.nchunks = min(nck, max(0, ncmax - chunk0));
      si.tok0 = tok0;
      si.len = len;
      smap[s] = si;
      if (N <= SORT_MAX) nckS[s] = nck;
    }
    __syncthreads();
    if (tid == 0) {
      int t = carry;
      for (int i = 0; i < NWAVE; ++i) t += wave_tot[i];
      carry = t;
    }
    __syncthreads();
  }
  for (int s = tid; s < N; s += NTHR) {
    int r = s;
    if (N <= SORT_MAX) {
      const int n = nckS[s];
      r = 0;
      for (int j = 0; j < N; ++j) {
        const int m = nckS[j];
        r += (m > n || (m == n && j < s)) ? 1 : 0;
      }
    }
    sorder[r] = s;
  }
}

// k_seg_map: the virtual sequence table of the segmented scans over packed
// sequences.  Segment p of sequence s is virtual row s P + p: chunks [p L,
// min((p + 1) L, n)) of the sequence's n chunks with L = ceil(n / P), empty
// past its end; one thread per virtual row.
__global__ __launch_bounds__(NTHR) void k_seg_map(const SeqInfo* __restrict__ smap, int N, int P,
                                                  SeqInfo* __restrict__ vmap) {
  const int i = blockIdx.x * NTHR + threadIdx.x;
  if (i >= N * P) return;
  const int s = i / P, p = i - s * P;
  const SeqInfo si = smap[s];
  const int L = (si.nchunks + P - 1) / P;
  const int c0 = min(p * L, si.nchunks), nc = min(L, si.nchunks - c0);
  SeqInfo v;
  v.chunk0 = si.chunk0 + c0;
  v.nchunks = nc;
  v.tok0 = si.tok0 + c0 * CH;
  v.len = nc > 0 ? min(si.len - c0 * CH, nc * CH) : 0;
  vmap[i] = v;
}

// k_chunk_fill: one thread per chunk slot c < ncmax.  Its sequence is the last
// one whose first chunk is <= c (first chunks never decrease, and an empty
// sequence shares its first chunk with the next one), found by binary search;
// slots past the last chunk are marked empty (len 0, seq -1).
__global__ __launch_bounds__(NTHR) void k_chunk_fill(const SeqInfo* __restrict__ smap, int N,
                                                     int ncmax, ChunkInfo* __restrict__ cmap) {
  for (int c = blockIdx.x * NTHR + threadIdx.x; c < ncmax; c += gridDim.x * NTHR) {
    int lo = 0, hi = N;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (smap[mid].chunk0 <= c) lo = mid + 1;
      else hi = mid;
    }
    ChunkInfo ci;
    ci.tok0 = 0;
    ci.len = 0;
    ci.seq = -1;
    ci.pad = 0;
    if (lo > 0) {
      const SeqInfo si = smap[lo - 1];
      const int j = c - si.chunk0;
      if (j < si.nchunks) {
        ci.tok0 = si.tok0 + j * CH;
        ci.len = min(CH, si.len - j * CH);
        ci.seq = lo - 1;
      }
    }
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
                                               const Tin* __restrict__ beta_tilde,
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

  {
    TileRegs<Tin, CH, DK> kr, qr;
    kr.load(k + tok * DK, (long)H * DK, ci.len);
    qr.load(q + tok * DK, (long)H * DK, ci.len);
    kr.store(Ks, LDK);
    qr.store(Qs, LDK);
  }
  if (w == 0) {
    const float gr = lane < ci.len ? g[tok + (long)lane * H] : 0.f;
    const float G = wave_prefix_sum(gr);
    Gs[lane] = G;
    Bs[lane] = lane < ci.len ? to_f(beta_tilde[tok + (long)lane * H]) : 0.f;  // feedback strength
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
    const Tin* __restrict__ beta, const Tin* __restrict__ beta_tilde, const float* __restrict__ d,
    const float* __restrict__ h0, const ChunkInfo* __restrict__ cmap,
    const SeqInfo* __restrict__ smap, int H, const float* __restrict__ Mw,
    const float* __restrict__ Aw, const float* __restrict__ Gw, float* __restrict__ o,
    float* __restrict__ ht, float* __restrict__ Xw, float* __restrict__ Dw) {
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
  __shared__ float Gs[CH], Bs[CH], Bts[CH];

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

  // registers holding the next chunk's tiles (loaded one chunk ahead)
  TileRegs<Tin, CH, DK> pk, pq;
  TileRegs<Tin, CH, BV> pv;
  TileRegs<float, CH, CH> pm, pa;
  float pg = 0.f, pb = 0.f, pbt = 0.f;
  auto issue = [&](int cc) {
    const int len = min(CH, si.len - cc * CH);
    const long chh = (long)(si.chunk0 + cc) * H + h;
    const long tok = (long)(si.tok0 + cc * CH) * H + h;
    pk.load(k + tok * DK, (long)H * DK, len);
    if constexpr (OUT) pq.load(q + tok * DK, (long)H * DK, len);
    pv.load(v + tok * DV + j0, (long)H * DV, len);
    pm.load(Mw + chh * CH * CH, CH, CH);
    if constexpr (OUT) pa.load(Aw + chh * CH * CH, CH, CH);
    if (threadIdx.x < CH) {
      const int r = threadIdx.x;
      pg = Gw[chh * CH + r];
      pb = r < len ? to_f(beta[tok + (long)r * H]) : 0.f;
      pbt = r < len ? to_f(beta_tilde[tok + (long)r * H]) : 0.f;
    }
  };
  if (si.nchunks > 0) issue(0);

  for (int cc = 0; cc < si.nchunks; ++cc) {
    const long chh = (long)(si.chunk0 + cc) * H + h;
    const long tok = (long)(si.tok0 + cc * CH) * H + h;
    ChunkInfo ci;
    ci.len = min(CH, si.len - cc * CH);
    __syncthreads();
    pk.store(Ks, LDK);
    pk.store_t(KsT, LDC);
    if constexpr (OUT) pq.store(Qs, LDK);
    pv.store(Vs, LDV);
    pm.store(Ms, LDF);
    if constexpr (OUT) pa.store(As, LDF);
    if (threadIdx.x < CH) {
      Gs[threadIdx.x] = pg;
      Bs[threadIdx.x] = pb;
      Bts[threadIdx.x] = pbt;
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
    if (cc + 1 < si.nchunks) issue(cc + 1);
    const float Glast = Gs[CH - 1];

    // K X and Q X for rows 16w..16w+15; R = Diag(beta) V - Diag(beta~ exp Gm) K X
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
        RT[jj * LDF + r] = Bs[r] * to_f(Vs[r * LDV + jj]) - Bts[r] * __expf(gm) * kxv;
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
    const Tin* __restrict__ beta_tilde, const float* __restrict__ d, const float* __restrict__ dht,
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

  TileRegs<Tin, CH, DK> pk, pq;
  TileRegs<Tin, CH, BV> pdo;
  TileRegs<float, CH, CH> pm, pa;
  float pg = 0.f, pb = 0.f;
  auto issue = [&](int cc) {
    const int len = min(CH, si.len - cc * CH);
    const long chh = (long)(si.chunk0 + cc) * H + h;
    const long tok = (long)(si.tok0 + cc * CH) * H + h;
    pk.load(k + tok * DK, (long)H * DK, len);
    pq.load(q + tok * DK, (long)H * DK, len);
    pdo.load(dO + tok * DV + j0, (long)H * DV, len);
    pa.load(Aw + chh * CH * CH, CH, CH);
    pm.load(Mw + chh * CH * CH, CH, CH);
    if (threadIdx.x < CH) {
      const int r = threadIdx.x;
      pg = Gw[chh * CH + r];
      pb = r < len ? to_f(beta_tilde[tok + (long)r * H]) : 0.f;
    }
  };
  if (si.nchunks > 0) issue(si.nchunks - 1);

  for (int cc = si.nchunks - 1; cc >= 0; --cc) {
    const long chh = (long)(si.chunk0 + cc) * H + h;
    __syncthreads();
    pk.store(Ks, LDK);
    pk.store_t(KsT, LDC);
    pq.store_t(QsT, LDC);
    pdo.store_t(dOT, LDC);
    pa.store_t(AsT, LDF);
    pm.store_t(MsT, LDF);
    if (threadIdx.x < CH) {
      Gs[threadIdx.x] = pg;
      Bs[threadIdx.x] = pb;
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
    if (cc > 0) issue(cc - 1);
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

    // dR = M^T dD;  Pg = Diag(exp G) dO;  W2 = -d Pg - Diag(beta~ exp Gm) dR
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
    const Tin* __restrict__ dO, const Tin* __restrict__ beta, const Tin* __restrict__ beta_tilde,
    const float* __restrict__ d, const ChunkInfo* __restrict__ cmap, int H,
    const float* __restrict__ Gw, const float* __restrict__ Xw, const float* __restrict__ Dw,
    const float* __restrict__ Yw, const float* __restrict__ dRw, float* __restrict__ dq,
    float* __restrict__ dk, float* __restrict__ dv, float* __restrict__ dbeta,
    float* __restrict__ dbeta_tilde, float* __restrict__ dg, float* __restrict__ ddp) {
  using SM = IntraBwdSmem<Tin, DK, DV>;
  constexpr bool F32 = is_f32<Tin>::value;
  constexpr int VB = SM::VB, LDK = SM::LDK, LDC = SM::LDC, LDVB = SM::LDVB, LDF = SM::LDF,
                LDFB = SM::LDFB;
  constexpr int NTK = DK / 16;
  __shared__ __align__(16) char smem[SM::BYTES];
  // rowB: derivative through beta (write strength), rowBt: through beta~
  // (feedback strength, in L and in R's K X term)
  __shared__ float Gs[CH], Bs[CH], Bts[CH], rowG[CH], rowGm[CH], rowB[CH], rowBt[CH];
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
    Bts[tid] = tid < len ? to_f(beta_tilde[tok + (long)tid * H]) : 0.f;
    rowG[tid] = 0.f;
    rowGm[tid] = 0.f;
    rowBt[tid] = 0.f;
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
  TileRegs<Tin, CH, VB> rdo, rv;
  TileRegs<float, CH, VB> rdr, rdl;
  TileRegs<float, DK, VB> rx, ry;
  auto issue = [&](int vb) {
    rdo.load(dO + tok * DV + vb * VB, (long)H * DV, len);
    rv.load(v + tok * DV + vb * VB, (long)H * DV, len);
    rdr.load(dRw + chh * CH * DV + vb * VB, DV, CH);
    rdl.load(Dw + chh * CH * DV + vb * VB, DV, CH);
    rx.load(Xw + chh * DK * DV + vb * VB, DV, DK);
    ry.load(Yw + chh * DK * DV + vb * VB, DV, DK);
  };
  issue(0);
  for (int vb = 0; vb < DV / VB; ++vb) {
    __syncthreads();
    rdo.store(dOb, LDVB);
    rv.store(Vb, LDVB);
    rdr.store(dRb, LDFB);
    rdl.store(Dlb, LDFB);
    rx.store(Xb, LDFB);
    ry.store(Yb, LDFB);
    __syncthreads();
    if (vb + 1 < DV / VB) issue(vb + 1);
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
  {
    TileRegs<Tin, CH, DK> kr, qr;
    kr.load(k + tok * DK, (long)H * DK, len);
    qr.load(q + tok * DK, (long)H * DK, len);
    kr.store(Ks, LDK);
    kr.store_t(KsT, LDC);
    qr.store(Qs, LDK);
    qr.store_t(QsT, LDC);
  }
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
          e2 = dl * Bts[r] * lck;
          rBL[e] += dl * lck;
          dakk = dl * Bts[r] * lc;
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
        rowBt[r] += rBL[e];
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
        rowGm[r] -= Bts[r] * egm * p3[e];
        rowBt[r] -= egm * p3[e];
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
      T2[0][nt][e] = __expf(Glast - Gs[r]) * T2[0][nt][e] - Bts[r] * egm * T3[0][nt][e];
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
      if (dbeta_tilde) {
        dbeta[tok + (long)r * H] = rowB[r];
        dbeta_tilde[tok + (long)r * H] = rowBt[r];
      } else {
        dbeta[tok + (long)r * H] = rowB[r] + rowBt[r];
      }
    }
    if (lane == 0) ddp[chh] = -dds;
  }
}

// dd[h] = sum over chunks of the per-chunk partials, one wave per head in a
// fixed order (lane l takes chunks l, l + 64, ..., then a butterfly over the
// wave): no LDS round trips or barriers
constexpr int RDD_THR = 64;
__global__ __launch_bounds__(RDD_THR) void k_reduce_dd(const float* __restrict__ ddp, int nc, int H,
                                                       float* __restrict__ dd) {
  const int h = blockIdx.x;
  float s = 0.f;
  for (int c = threadIdx.x; c < nc; c += RDD_THR) s += ddp[(long)c * H + h];
  s = wave_sum(s);
  if (threadIdx.x == 0) dd[h] = s;
}

// ===========================================================================
// bf16 path.  k_prep_bf writes the per-chunk operands the scans need in the
// order the MFMA consumes them: M and A as int16 with one power-of-two scale
// per row of M and per column of A, and for the backward Q^T as bf16.  In the
// forward scan each wave loads the fragments of its own rows straight from
// global memory into registers, one chunk ahead; LDS carries what the four
// waves exchange (state, R, D and their backward counterparts, already split)
// and the chunk's K rows, whose transposing reads give the K^T operand.  The
// reverse scan stages the same M and A fragments in LDS and reads M^T, A^T
// back with transposing reads.
// ===========================================================================
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// dv columns per scan workgroup: a chain (sequence, head) is split into
// dv / SCAN_BV independent workgroups
#ifndef COMBA_SCAN_BV
#define COMBA_SCAN_BV 32
#endif
constexpr int SCAN_BV = COMBA_SCAN_BV;

__device__ __forceinline__ floatx4 mfma16(const bf16x8& a, const bf16x8& b, const floatx4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ bf16x8 ld8(const bf16_t* p) { return *reinterpret_cast<const bf16x8*>(p); }
__device__ __forceinline__ bf16x8 zero8() { return __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u}); }

// Chunk and sequence tables of the bf16 kernels: for fixed-length rows
// (Tfix >= 0 tokens each) in closed form, for packed sequences (Tfix < 0) from
// the tables of k_seq_map and k_chunk_fill.
__device__ __forceinline__ ChunkInfo chunk_at(const ChunkInfo* cmap, int c, int Tfix) {
  if (Tfix >= 0) {
    const int ncs = max(1, (Tfix + CH - 1) / CH), s = c / ncs, i = c - s * ncs;
    return ChunkInfo{s * Tfix + i * CH, min(CH, Tfix - i * CH), s, 0};
  }
  return cmap[c];
}
__device__ __forceinline__ SeqInfo seq_at(const SeqInfo* smap, int s, int Tfix) {
  if (Tfix >= 0) {
    const int ncs = (Tfix + CH - 1) / CH;
    return SeqInfo{s * ncs, ncs, s * Tfix, Tfix};
  }
  return smap[s];
}

// Element (row, col) of a 64-column operand tile that prep stores in MFMA
// fragment order (M, A, Q^T): the 16 bytes lane (g, i) of wave w
// loads for k-step ks (row 16 w + i, columns 32 ks + 8 g .. +7) sit at
// ((2 (row / 16) + ks) 64 + 16 g + i) * 8, so one k-step load of a wave reads
// 1 KiB of whole lines (a row-major fragment would touch 16 half lines).
__device__ __forceinline__ int frag_off(int row, int col) {
  return (((row >> 4) * 2 + (col >> 5)) * 64 + ((col >> 3) & 3) * 16 + (row & 15)) * 8 + (col & 7);
}

// Workgroup -> (sequence s, head h, dv slice zb) of the bf16 scans (a 1-D grid of
// scan_blocks workgroups).  The NSL slices of one (sequence, head) chain are
// workgroups 8 NSL g + 8 zb + c8: their indices agree mod 8, so the round-robin
// dispatch puts them on the same XCD, and they are dispatched together, so the
// K, Q, M, A rows they all read are L2 hits for all but the first.  Chains are
// taken rank-major (r = chain / H), with packed sequences in the order of
// sorder (longest first); padding workgroups past the last chain return.
// grp > 1 (the segmented scans' state passes): the rows are groups of grp
// segments of which one is skipped (the last, goff = 0, or the first, goff =
// 1), so rank r is row (r / (grp - 1)) grp + goff + r % (grp - 1) and N counts
// the rows taken.
template <int NSL>
__device__ __forceinline__ bool scan_item(int N, int H, const int* sorder, int& s, int& h, int& zb,
                                          int grp = 0, int goff = 0) {
  const int L = blockIdx.x;
  zb = (L >> 3) % NSL;
  const int chain = (L / (8 * NSL)) * 8 + (L & 7);
  if (chain >= N * H) return false;
  const int r = chain / H;
  h = chain - r * H;
  s = sorder ? sorder[r] : grp > 1 ? (r / (grp - 1)) * grp + goff + r % (grp - 1) : r;
  return true;
}

// four fp32 values -> bf16 (hi, lo) with hi + lo ~ x to ~16 significant bits
__device__ __forceinline__ void split4(const float (&x)[4], bf16x4& hi, bf16x4& lo) {
  uint32_t h0, h1, l0, l1;
  split2(x[0], x[1], h0, l0);
  split2(x[2], x[3], h1, l1);
  hi = __builtin_bit_cast(bf16x4, make_uint2(h0, h1));
  lo = __builtin_bit_cast(bf16x4, make_uint2(l0, l1));
}
// store the 4 values a lane holds in one accumulator column (rows 4g..4g+3)
// into a transposed, split LDS buffer: dst[col * ld + row0 + e]
__device__ __forceinline__ void put_t4(bf16_t* hi, bf16_t* lo, int off, const float (&x)[4]) {
  bf16x4 h, l;
  split4(x, h, l);
  *reinterpret_cast<bf16x4*>(hi + off) = h;
  *reinterpret_cast<bf16x4*>(lo + off) = l;
}

// Block column J of M = (I + L)^{-1} below the diagonal, in the accumulator
// layout of the 16x16 fp32 MFMA: on entry mb[J] = D_J; on exit mb[i] = M_iJ for
// i > J.  The L_ik and D_i blocks come from LDS (row-major, stride LDL, D_i in
// the diagonal blocks).  Each product runs its k index in the order
// 4 (lane / 16) + e at step e, so that an accumulator is directly the B operand
// of the next product and the A operand of a step is one 16-byte LDS read.
template <int J, int LDL>
__device__ __forceinline__ void solve_block_column(const float* Ls, floatx4 (&mb)[4]) {
  const int lane = lane_id(), r16 = lane & 15, g4 = lane >> 4;
#pragma unroll
  for (int i = J + 1; i < 4; ++i) {
    floatx4 t = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = J; kb < i; ++kb) {
      const float4 a = *reinterpret_cast<const float4*>(Ls + (16 * i + r16) * LDL + 16 * kb + 4 * g4);
      t = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, mb[kb][0], t, 0, 0, 0);
      t = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, mb[kb][1], t, 0, 0, 0);
      t = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, mb[kb][2], t, 0, 0, 0);
      t = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, mb[kb][3], t, 0, 0, 0);
    }
    const float4 dd = *reinterpret_cast<const float4*>(Ls + (16 * i + r16) * LDL + 16 * i + 4 * g4);
    floatx4 u = {0.f, 0.f, 0.f, 0.f};
    u = __builtin_amdgcn_mfma_f32_16x16x4f32(dd.x, t[0], u, 0, 0, 0);
    u = __builtin_amdgcn_mfma_f32_16x16x4f32(dd.y, t[1], u, 0, 0, 0);
    u = __builtin_amdgcn_mfma_f32_16x16x4f32(dd.z, t[2], u, 0, 0, 0);
    u = __builtin_amdgcn_mfma_f32_16x16x4f32(dd.w, t[3], u, 0, 0, 0);
    mb[i] = -u;
  }
}

// Block column J of M (mb as left by solve_block_column) into LDS over L.
template <int J, int LDL>
__device__ __forceinline__ void put_block_column(float* Ls, const floatx4 (&mb)[4]) {
  const int lane = lane_id(), r16 = lane & 15, g4 = lane >> 4;
#pragma unroll
  for (int i = J + 1; i < 4; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) Ls[(16 * i + 4 * g4 + e) * LDL + 16 * J + r16] = mb[i][e];
}

template <int DK, bool BWD>
__global__ __launch_bounds__(NTHR) void k_prep_bf(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ k, const float* __restrict__ g,
    const bf16_t* __restrict__ beta_tilde, const float* __restrict__ d,
    const ChunkInfo* __restrict__ cmap, int Tfix, int H, int16_t* __restrict__ Mq, float* __restrict__ Ms, int16_t* __restrict__ Aq,
    float* __restrict__ As, bf16_t* __restrict__ QTp, float* __restrict__ Gw) {
  // M leaves as int16 with one power-of-two scale per row, A with one per
  // column (see q_pack4).  The forward scan takes M's row scale out of the
  // rows of M R and folds A's column scale into the matching rows of D before
  // A D; the reverse scan reads both tiles transposed (M^T dD, A^T dO), folds
  // M's row scale into the rows of dD and takes A's column scale out of the
  // rows of A^T dO.  With BWD it also stores Q^T for the reverse scan.
  constexpr int LDK = DK + 24;  // 304-byte rows: conflict-free 16-byte and transposing reads
  constexpr int LDL = CH + 4;
  constexpr int CC = CH * CH;
  // the Q tile is dead once K^T, Q^T and Q K^T are taken: L (then M) reuses
  // its LDS, which keeps four workgroups on a CU
  constexpr int QLB = CH * LDL * 4 > CH * LDK * 2 ? CH * LDL * 4 : CH * LDK * 2;
  __shared__ __align__(16) bf16_t Ks[CH * LDK];
  __shared__ __align__(16) unsigned char QLbuf[QLB];
  bf16_t* Qs = reinterpret_cast<bf16_t*>(QLbuf);
  float* Ls = reinterpret_cast<float*>(QLbuf);
  __shared__ float Gs[CH], Bs[CH];
  __shared__ float colmax[NWAVE][CH];  // per-wave column maxima of |A|

  const ChunkInfo ci = chunk_at(cmap, blockIdx.x, Tfix);
  if (ci.len <= 0) return;
  const int h = blockIdx.y;
  const long chh = (long)blockIdx.x * H + h;
  const long tok = (long)ci.tok0 * H + h;
  const int w = wave_id(), lane = lane_id(), g4 = lane >> 4, r16 = lane & 15;
  const float dh = d[h];
  {
    // every load is unconditional (clamped rows, zeroed where used): a branch
    // around a load makes the wave wait for it on the spot
    const long grow = tok + (long)min(lane, ci.len - 1) * H;
    const float g_in = g[grow], b_in = bf2f(beta_tilde[grow]);  // feedback strength (L only)
    TileRegs<bf16_t, CH, DK> kr, qr;
    kr.load_clip(k + tok * DK, (long)H * DK, ci.len);
    qr.load_clip(q + tok * DK, (long)H * DK, ci.len);
    // every wave forms G and writes the same Gs, Bs (no branch around the uses)
    const float G = wave_prefix_sum(lane < ci.len ? g_in : 0.f);
    Gs[lane] = G;
    Bs[lane] = lane < ci.len ? b_in : 0.f;
    if (w == 0) Gw[chh * CH + lane] = G;
    kr.store(Ks, LDK);
    qr.store(Qs, LDK);
  }
  __syncthreads();
  if constexpr (BWD) {
    // Q^T per chunk-head, dk x 64 bf16 in fragment order, for the reverse scan.  One transposing
    // LDS read pair gives lane (g, i) the 8 rows 32 tb + 8 g .. of column c0 + i,
    // i.e. one 16-byte piece of row c0 + i of Q^T.
    bf16_t* Qt = QTp + chh * DK * CH;
    for (int pc = w; pc < 2 * (DK / 16); pc += NWAVE) {
      const int c0 = 16 * (pc % (DK / 16)), r0 = 32 * (pc / (DK / 16)) + 8 * g4;
      *reinterpret_cast<bf16x8*>(Qt + frag_off(c0 + (lane & 15), r0)) = ld_tr8(Qs, LDK, r0, c0);
    }
  }

  floatx4 akk[1][4], aqk[1][4];
  zero_acc(akk);
  zero_acc(aqk);
  mma<false, 1, 4, DK>(akk, Ks + 16 * w * LDK, LDK, Ks, LDK);
  mma<false, 1, 4, DK>(aqk, Qs + 16 * w * LDK, LDK, Ks, LDK);
  __syncthreads();  // every read of the Q tile is done: L overwrites it
  // A in the accumulator layout: av[nt][e] = A[16w + 4g4 + e][16nt + r16]
  float av[4][4];
#pragma unroll
  for (int nt = 0; nt < 4; ++nt) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = 16 * w + acc_row(0, e), c = acc_col(nt);
      const float kk = akk[0][nt][e];
      float a = 0.f, l = 0.f;
      if (r >= c) a = (aqk[0][nt][e] - dh * kk) * __expf(Gs[r] - Gs[c]);
      if (r > c) l = Bs[r] * __expf(Gs[r - 1] - Gs[c]) * kk;
      av[nt][e] = a;
      Ls[r * LDL + c] = l;
    }
  }
  // column maxima of this wave's 16 rows, combined over the waves below
#pragma unroll
  for (int nt = 0; nt < 4; ++nt) {
    float m = nmax_abs4(0.f, floatx4{av[nt][0], av[nt][1], av[nt][2], av[nt][3]});
    m = nmax(m, __shfl_xor(m, 16));
    m = nmax(m, __shfl_xor(m, 32));
    if (g4 == 0) colmax[w][16 * nt + r16] = m;
  }
  __syncthreads();
  {
    auto col_max = [&](int c) {
      return nmax(nmax(colmax[0][c], colmax[1][c]), nmax(colmax[2][c], colmax[3][c]));
    };
    // A rows leave as 8-byte pieces of four columns (see quad_transpose): the
    // lane's row after the transpose is 16w + qt_row(), its columns
    // 16nt + qt_col() .. +3, each with its own column scale
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      const int c0 = 16 * nt + qt_col();
      const floatx4 inv = {q_inv_scale(col_max(c0)), q_inv_scale(col_max(c0 + 1)),
                           q_inv_scale(col_max(c0 + 2)), q_inv_scale(col_max(c0 + 3))};
      *reinterpret_cast<uint2*>(Aq + chh * CC + frag_off(16 * w + qt_row(), c0)) =
          q_pack4v(quad_transpose(floatx4{av[nt][0], av[nt][1], av[nt][2], av[nt][3]}), inv);
    }
    if (w == 0) As[chh * CH + lane] = q_scale(col_max(lane));
  }

  // M = (I + L)^{-1} by 16x16 blocks (L is strictly lower triangular, so M is
  // unit lower triangular).  Wave w owns block column jb: it inverts the
  // diagonal block, D_jb = (I + L_jb,jb)^{-1}, then walks down its block column
  // with M_ij = -D_i sum_{j <= k < i} L_ik M_kj.  Block columns do not depend
  // on one another; the rotation spreads the longest column (jb = 0) over the
  // SIMDs of workgroups that share a CU.
  const int jb = (w + blockIdx.x + blockIdx.y) & (NWAVE - 1);
  floatx4 mb[4];
  {
    // lane (g4, r16) solves column r16 of the diagonal block by forward
    // substitution in fp32 (the four 16-lane groups redundantly)
    float* Lb = Ls + 16 * jb * LDL + 16 * jb;
    float x[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) x[i] = (i == r16) ? 1.f : 0.f;
#pragma unroll
    for (int i = 1; i < 16; ++i) {
      float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
#pragma unroll
      for (int m = 0; m < i; m += 4) {
        const float4 lv = *reinterpret_cast<const float4*>(Lb + i * LDL + m);
        s0 += lv.x * x[m];
        if (m + 1 < i) s1 += lv.y * x[m + 1];
        if (m + 2 < i) s2 += lv.z * x[m + 2];
        if (m + 3 < i) s3 += lv.w * x[m + 3];
      }
      if (i > r16) x[i] = -((s0 + s1) + (s2 + s3));
    }
    // D_jb in the accumulator layout (rows 4 g4 + e of column r16) replaces
    // L_jb,jb in LDS; only this wave reads that block, and its reads are done
    floatx4 dm;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      dm[e] = g4 == 0 ? x[e] : g4 == 1 ? x[4 + e] : g4 == 2 ? x[8 + e] : x[12 + e];
      Lb[(4 * g4 + e) * LDL + r16] = dm[e];
    }
    mb[0] = mb[1] = mb[2] = mb[3] = dm;
  }
  __syncthreads();
  switch (jb) {
    case 0: solve_block_column<0, LDL>(Ls, mb); break;
    case 1: solve_block_column<1, LDL>(Ls, mb); break;
    case 2: solve_block_column<2, LDL>(Ls, mb); break;
    default: break;
  }
  __syncthreads();  // every read of L is done
  switch (jb) {
    case 0: put_block_column<0, LDL>(Ls, mb); break;
    case 1: put_block_column<1, LDL>(Ls, mb); break;
    case 2: put_block_column<2, LDL>(Ls, mb); break;
    default: put_block_column<3, LDL>(Ls, mb); break;
  }
  __syncthreads();
  // M rows from LDS as 16-byte pieces of eight columns; the 8 threads of a row
  // are one 8-lane group, which reduces the row maximum
  static_assert(CC / 8 % NTHR == 0, "every thread takes whole passes");
  for (int idx = threadIdx.x; idx < CC / 8; idx += NTHR) {
    const int r = idx / (CH / 8), c8 = (idx % (CH / 8)) * 8;
    const float4 m0 = *reinterpret_cast<const float4*>(Ls + r * LDL + c8);
    const float4 m1 = *reinterpret_cast<const float4*>(Ls + r * LDL + c8 + 4);
    const float mv[8] = {m0.x, m0.y, m0.z, m0.w, m1.x, m1.y, m1.z, m1.w};
    float m = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) m = nmax(m, fabsf(mv[e]));
    m = max8(m);
    *reinterpret_cast<uint4*>(Mq + chh * CC + frag_off(r, c8)) = q_pack8(mv, q_inv_scale(m));
    Ms[chh * CH + r] = q_scale(m);  // the eight threads of a row store the same value
  }
}

// Forward state scan (bf16 inputs).  One workgroup per (sequence, head,
// 32-wide dv slice); wave w owns rows 16w..16w+15 of the chunk products and
// rows (dk/4)w.. of the state slice.  Every product is formed transposed (the
// MFMA operands swapped), so that an accumulator gives a lane one row and four
// consecutive columns: rows leave for memory as they are (no transposes), a
// lane needs the gates and beta of one row only, and the intermediate tiles
// (state, R, D, Dg) sit row-major in LDS, read as operands with transposing
// reads.
// PHI: the homogeneous recurrence from the identity (no value term, X_0 = I,
// DV = DK columns): the final state is the product of the chunks' transitions
// X -> e^{G_63} X - K~^T M Diag(s) K X over the sequence (the segment
// transition of the segmented scan, run_fwd_bf).
template <int DK, int DV, int BV, bool OUT, bool STORE, bool PHI = false>
__global__ __launch_bounds__(NTHR, 1) void k_scan_fwd_bf(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ k, const bf16_t* __restrict__ v,
    const bf16_t* __restrict__ beta, const bf16_t* __restrict__ beta_tilde,
    const float* __restrict__ d, const float* __restrict__ h0,
    const SeqInfo* __restrict__ smap, const int* __restrict__ sorder, int N, int Tfix, int H,
    const int16_t* __restrict__ Mq,
    const float* __restrict__ Ms, const int16_t* __restrict__ Aq, const float* __restrict__ As,
    const float* __restrict__ Gw, float* __restrict__ o, float* __restrict__ ht, int16_t* __restrict__ Xq,
    float* __restrict__ Xs, int16_t* __restrict__ Dq, float* __restrict__ Ds,
    int16_t* __restrict__ Xfq, float* __restrict__ Xfs, int grp = 0) {
  // Every global load and store inside the chunk loop is issued unconditionally
  // (clamped rows and chunk indices, masked values applied at use, padded-row
  // stores dropped by the record count of a raw buffer), so the memory-counter
  // waits stay exact and the next chunk's loads overlap the current chunk's work.
  constexpr int NTV = BV / 16, XMT = DK / 64, KS = DK / 32, CC = CH * CH;
  constexpr int NB = DV / 32;
  // row-major BV-wide tiles: 72-byte rows put the four rows of a transposing
  // read on disjoint banks
  constexpr int LDT = BV + 4;
  static_assert(BV == 32, "stored states use one scale per 32-column block = one dv slice");
  static_assert(!PHI || (DV == DK && !OUT && !STORE), "the transition product is a dk x dk state");
  __shared__ __align__(16) bf16_t Xh[DK * LDT];
  __shared__ __align__(16) bf16_t Xl[DK * LDT];
  __shared__ __align__(16) bf16_t Rh[CH * LDT];
  __shared__ __align__(16) bf16_t Rl[CH * LDT];
  __shared__ __align__(16) bf16_t Dgh[CH * LDT];
  __shared__ __align__(16) bf16_t Dgl[CH * LDT];
  __shared__ __align__(16) bf16_t Dh[OUT ? CH * LDT : 8];
  __shared__ __align__(16) bf16_t Dl[OUT ? CH * LDT : 8];
  // the chunk's K rows, staged from the K operand registers: the state update
  // takes its K operand (reduction down the chunk rows) from here with
  // transposing reads
  constexpr int LDKC = DK + 24;  // 304-byte rows: conflict-free transposing reads
  __shared__ __align__(16) bf16_t Kc[CH * LDKC];

  int s, h, zb;
  if (!scan_item<DV / BV>(N, H, sorder, s, h, zb, grp)) return;
  const int j0 = zb * BV;
  const SeqInfo si = seq_at(smap, s, Tfix);
  const int w = wave_id(), lane = lane_id(), r16 = lane & 15, g4 = lane >> 4;
  const long soff = ((long)s * H + h) * DK * DV;
  const float dh = d[h];
  const int n = si.nchunks;
  const int prow = 16 * w + r16;            // chunk row of this lane
  const int xrow0 = (DK / 4) * w + r16;     // state rows of this lane: xrow0 + 16 mt
  const int col0 = 4 * g4;                  // columns of this lane: 16 nt + col0 .. +3

  // state, accumulator layout of the transposed products: row xrow0 + 16 mt,
  // columns 16 nt + col0 .. +3 of the slice
  floatx4 X[XMT][NTV];
#pragma unroll
  for (int mt = 0; mt < XMT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NTV; ++nt) {
      if constexpr (PHI) {
        const int r = xrow0 + 16 * mt, c = j0 + 16 * nt + col0;
#pragma unroll
        for (int e = 0; e < 4; ++e) X[mt][nt][e] = r == c + e ? 1.f : 0.f;
      } else if (h0) {
        const float4 x4 = *reinterpret_cast<const float4*>(h0 + soff + (long)(xrow0 + 16 * mt) * DV + j0 + 16 * nt + col0);
        X[mt][nt] = floatx4{x4.x, x4.y, x4.z, x4.w};
      } else {
        X[mt][nt] = zero4();
      }
    }
  auto put_state = [&]() {
#pragma unroll
    for (int mt = 0; mt < XMT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt) {
        const float xv[4] = {X[mt][nt][0], X[mt][nt][1], X[mt][nt][2], X[mt][nt][3]};
        put_t4(Xh, Xl, (xrow0 + 16 * mt) * LDT + 16 * nt + col0, xv);
      }
  };
  auto store_state = [&](float* dst) {
#pragma unroll
    for (int mt = 0; mt < XMT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt)
        store4(dst + (long)(xrow0 + 16 * mt) * DV + j0 + 16 * nt + col0, X[mt][nt]);
  };
  // The same rows as int16 with one scale per row of the slice (see q_pack4),
  // into the slice's own block: dq = block base, [DK][BV]; ds = its row scales.
  // A row's 32 columns are spread over the four lanes r16 + 16 g4; they are
  // regrouped so that each lane stores 16 bytes (row8_from_pieces), and lane
  // group g4 stores the scale of row xrow0 + 16 g4 (one store for all rows).
  auto store_state_q = [&](int16_t* dq, float* ds) {
    float sc = 0.f;
#pragma unroll
    for (int mt = 0; mt < XMT; ++mt) {
      float m = nmax_abs4(nmax_abs4(0.f, X[mt][0]), X[mt][1]);
      m = rowgroup_max(m);
      const float inv = q_inv_scale(m);
      const unsigned row = xrow0 + 16 * mt;
      at(reinterpret_cast<uint4*>(dq), 2u * (row * BV + row8_col())) =
          row8_from_pieces(q_pack4(X[mt][0], inv), q_pack4(X[mt][1], inv));
      if (g4 == mt) sc = q_scale(m);
    }
    if (g4 < XMT) at(ds, 4u * (xrow0 + 16 * g4)) = sc;
  };
  put_state();

  // chunk offsets are wave-uniform; readfirstlane keeps them (and every chunk
  // base address) in scalar registers, so that loads and stores take a scalar
  // base and a 32-bit lane offset
  auto c_len = [&](int cc) { return min(CH, si.len - cc * CH); };
  auto c_tok = [&](int cc) { return (long)__builtin_amdgcn_readfirstlane(si.tok0 + cc * CH) * H + h; };
  auto c_chh = [&](int cc) { return (long)__builtin_amdgcn_readfirstlane(si.chunk0 + cc) * H + h; };

  // per-chunk operands, loaded one chunk ahead: K, Q rows as bf16, the rows of
  // M and A as int16 with M's row scale (applied to the accumulator rows:
  // (M R)[r] = s_r sum_i q[r][i] R[i]) and A's column scale (applied to the
  // rows of D before A D: (A D)[r] = sum_c q[r][c] (s_c D[c]))
  bf16x8 kf[KS], qf[KS];
  uint4 mq[2], aq[2];
  float msc, asc;
  // per-row values of the chunk (cumulative gates G, beta, beta~, the V slice)
  // are loaded one chunk ahead into registers and staged through a
  // double-buffered LDS area at the end of each chunk
  __shared__ float Grow[2][CH], Brow[2][CH], BTrow[2][CH];
  __shared__ __align__(16) bf16_t Vrow[2][CH * (BV + 8)];
  constexpr int VPR = BV / 8;                  // 16-byte pieces per V row
  const int vr = threadIdx.x / VPR, vc = (threadIdx.x % VPR) * 8;
  const int vr_ld = min(vr, CH - 1);
  float pgv = 0.f;
  bf16_t pbv = 0, pbtv = 0;
  uint4 pvv = make_uint4(0, 0, 0, 0);
  int plen = 0;
  auto load_rows = [&](int cc) {
    plen = c_len(cc);
    const long tok = c_tok(cc), chh = c_chh(cc);
    const int t = threadIdx.x & (CH - 1);
    // chunk bases are wave-uniform (scalar registers), lane offsets 32-bit
    const unsigned tr = 2u * ((unsigned)min(t, plen - 1) * H);
    pgv = at(Gw + chh * CH, 4u * t);
    pbv = at(beta + tok, tr);
    pbtv = at(beta_tilde + tok, tr);
    if constexpr (!PHI)
      pvv = at(reinterpret_cast<const uint4*>(v + tok * DV + j0),
               2u * ((unsigned)min(vr_ld, plen - 1) * (H * DV) + vc));
  };
  auto put_rows = [&](int buf) {
    const int t = threadIdx.x & (CH - 1);
    Grow[buf][t] = pgv;
    // no value term in the transition product
    Brow[buf][t] = !PHI && t < plen ? bf2f(pbv) : 0.f;
    BTrow[buf][t] = t < plen ? bf2f(pbtv) : 0.f;
    if (CH * VPR >= NTHR || threadIdx.x < CH * VPR)
      *reinterpret_cast<uint4*>(&Vrow[buf][vr * (BV + 8) + vc]) =
          vr < plen ? pvv : make_uint4(0, 0, 0, 0);
  };
  // rows past the chunk end load a valid row; their K X / Q X results are
  // never used (beta = beta~ = 0 zeroes R there and such outputs are not stored)
  auto load_kq = [&](int cc) {
    const long tb = c_tok(cc) * DK;
    const unsigned rb = 2u * ((unsigned)min(prow, c_len(cc) - 1) * (H * DK) + 8 * g4);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      kf[ks] = at(reinterpret_cast<const bf16x8*>(k + tb), rb + 64u * ks);
      if constexpr (OUT) qf[ks] = at(reinterpret_cast<const bf16x8*>(q + tb), rb + 64u * ks);
    }
  };
  const unsigned foff = 16u * (2 * w * 64 + lane);  // this lane's fragment (fragment order)
  auto load_m = [&](int cc) {
    const uint4* p = reinterpret_cast<const uint4*>(Mq + c_chh(cc) * CC);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) mq[ks] = at(p, foff + 1024u * ks);
    msc = at(Ms + c_chh(cc) * CH, 4u * prow);
  };
  auto load_a = [&](int cc) {
    const uint4* p = reinterpret_cast<const uint4*>(Aq + c_chh(cc) * CC);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) aq[ks] = at(p, foff + 1024u * ks);
    asc = at(As + c_chh(cc) * CH, 4u * prow);
  };
  if (n > 0) {
    load_kq(0);
    load_m(0);
    if constexpr (OUT) load_a(0);
    load_rows(0);
    put_rows(0);
  }
  __syncthreads();

  for (int cc = 0; cc < n; ++cc) {
    const bool more = cc + 1 < n;
    const int nx = more ? cc + 1 : cc;  // chunk prefetched during this one
    const int len = c_len(cc);
    const long tok = c_tok(cc), chh = c_chh(cc);
    const int buf = cc & 1;
    load_rows(nx);
    const float glast = Grow[buf][CH - 1];
    const float gg = Grow[buf][prow], gm = prow > 0 ? Grow[buf][prow - 1] : 0.f, bb = Brow[buf][prow];
    const float bt = BTrow[buf][prow];

    // (K X)^T and (Q X)^T: this lane holds row prow, columns 16 nt + col0 ..;
    // R = Diag(beta) V - Diag(beta~ exp Gm) K X
    floatx4 kx[NTV], qx[NTV];
#pragma unroll
    for (int nt = 0; nt < NTV; ++nt) {
      kx[nt] = zero4();
      qx[nt] = zero4();
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt) {
        const bf16x8 xh = ld_tr8(Xh, LDT, 32 * ks + 8 * g4, 16 * nt);
        const bf16x8 xl = ld_tr8(Xl, LDT, 32 * ks + 8 * g4, 16 * nt);
        kx[nt] = mfma16(xh, kf[ks], kx[nt]);
        kx[nt] = mfma16(xl, kf[ks], kx[nt]);
        if constexpr (OUT) {
          qx[nt] = mfma16(xh, qf[ks], qx[nt]);
          qx[nt] = mfma16(xl, qf[ks], qx[nt]);
        }
      }
    // the state entering this chunk, stored while the products above run
    // (stores bunched before a barrier stall all four waves at once)
    if constexpr (STORE) {
      const long xb = (chh * NB + zb) * DK;
      store_state_q(Xq + xb * BV, Xs + xb);
    }
    // K rows past the chunk end repeat row len - 1; D is zero there
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) *reinterpret_cast<bf16x8*>(Kc + prow * LDKC + 32 * ks + 8 * g4) = kf[ks];
    load_kq(nx);
    floatx4 oacc[NTV];
    {
      const float btegm = bt * __expf(gm), eg = __expf(gg);
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt) {
        const uint2 v4 = *reinterpret_cast<const uint2*>(&Vrow[buf][prow * (BV + 8) + 16 * nt + col0]);
        const float vv[4] = {__uint_as_float(v4.x << 16), __uint_as_float(v4.x & 0xFFFF0000u),
                             __uint_as_float(v4.y << 16), __uint_as_float(v4.y & 0xFFFF0000u)};
        float rv[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          rv[e] = bb * vv[e] - btegm * kx[nt][e];
          if constexpr (OUT) oacc[nt][e] = eg * (qx[nt][e] - dh * kx[nt][e]);
        }
        put_t4(Rh, Rl, prow * LDT + 16 * nt + col0, rv);
      }
    }
    __syncthreads();

    // (M R)^T
    floatx4 dl[NTV];
#pragma unroll
    for (int nt = 0; nt < NTV; ++nt) dl[nt] = zero4();
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      bf16x8 mh, ml;
      q_split8(mq[ks], mh, ml);
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt) {
        const bf16x8 rh = ld_tr8(Rh, LDT, 32 * ks + 8 * g4, 16 * nt);
        const bf16x8 rl = ld_tr8(Rl, LDT, 32 * ks + 8 * g4, 16 * nt);
        dl[nt] = mfma16(rh, mh, dl[nt]);
        dl[nt] = mfma16(rl, mh, dl[nt]);
        dl[nt] = mfma16(rh, ml, dl[nt]);
      }
    }
    const float ms_cur = msc;
    load_m(nx);
#pragma unroll
    for (int nt = 0; nt < NTV; ++nt) dl[nt] *= ms_cur;
    // D rows as int16 with one scale per row of the slice, stored after the
    // next phase's products are issued
    uint4 dpk = make_uint4(0u, 0u, 0u, 0u);
    float dsc = 0.f;
    if constexpr (STORE) {
      const float m = rowgroup_max(nmax_abs4(nmax_abs4(0.f, dl[0]), dl[1]));
      const float inv = q_inv_scale(m);
      dpk = row8_from_pieces(q_pack4(dl[0], inv), q_pack4(dl[1], inv));
      dsc = q_scale(m);
    }
    {
      const float edec = __expf(glast - gg);
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt) {
        const float dv[4] = {dl[nt][0], dl[nt][1], dl[nt][2], dl[nt][3]};
        const float dgv[4] = {edec * dv[0], edec * dv[1], edec * dv[2], edec * dv[3]};
        const int off = prow * LDT + 16 * nt + col0;
        put_t4(Dgh, Dgl, off, dgv);
        if constexpr (OUT) {
          // times A's column scale for column prow (a power of two: exact)
          const float dav[4] = {asc * dv[0], asc * dv[1], asc * dv[2], asc * dv[3]};
          put_t4(Dh, Dl, off, dav);
        }
      }
    }
    __syncthreads();

    // X'^T = exp(G_63) X^T + (Diag(exp(G_63 - G)) D)^T K
    const float gC = __expf(glast);
#pragma unroll
    for (int mt = 0; mt < XMT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt) X[mt][nt] *= gC;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      // K fragments for state rows (dk/4) w + 16 mt + r16, chunk rows 32 ks + 8 g4 ..
      bf16x8 ktf[XMT];
#pragma unroll
      for (int mt = 0; mt < XMT; ++mt) ktf[mt] = ld_tr8(Kc, LDKC, 32 * ks + 8 * g4, (DK / 4) * w + 16 * mt);
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt) {
        const bf16x8 dgh = ld_tr8(Dgh, LDT, 32 * ks + 8 * g4, 16 * nt);
        const bf16x8 dgl = ld_tr8(Dgl, LDT, 32 * ks + 8 * g4, 16 * nt);
#pragma unroll
        for (int mt = 0; mt < XMT; ++mt) {
          X[mt][nt] = mfma16(dgh, ktf[mt], X[mt][nt]);
          X[mt][nt] = mfma16(dgl, ktf[mt], X[mt][nt]);
        }
      }
    }
    if constexpr (STORE) {
      const long blk = (chh * NB + zb) * CH;  // the slice's block
      at(reinterpret_cast<uint4*>(Dq + blk * BV), 2u * (prow * BV + row8_col())) = dpk;
      if (g4 == 0) at(Ds + blk, 4u * prow) = dsc;
    }

    // O = Diag(exp G)(Q - d K) X + A D, formed as (A D)^T = D^T A^T
    if constexpr (OUT) {
      floatx4 adc[NTV];
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt) adc[nt] = zero4();
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        bf16x8 ah, al;
        q_split8(aq[ks], ah, al);
#pragma unroll
        for (int nt = 0; nt < NTV; ++nt) {
          const bf16x8 dh_ = ld_tr8(Dh, LDT, 32 * ks + 8 * g4, 16 * nt);
          const bf16x8 dl_ = ld_tr8(Dl, LDT, 32 * ks + 8 * g4, 16 * nt);
          adc[nt] = mfma16(dh_, ah, adc[nt]);
          adc[nt] = mfma16(dl_, ah, adc[nt]);
          adc[nt] = mfma16(dh_, al, adc[nt]);
        }
      }
      load_a(nx);
      // rows past the chunk end fall past the record count: dropped
      const __amdgpu_buffer_rsrc_t ro = clip_rsrc(o + tok * DV + j0, (unsigned)len * (unsigned)(H * DV * 4));
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt) {
        floatx4 ov;
#pragma unroll
        for (int e = 0; e < 4; ++e) ov[e] = oacc[nt][e] + adc[nt][e];
        store_clip4(ov, ro, 4u * ((unsigned)prow * (H * DV) + 16 * nt + col0));
      }
    }
    put_state();
    put_rows(buf ^ 1);
    __syncthreads();
  }
  // the state after the last chunk (the backward's sink for it; none in the
  // segmented scan)
  if constexpr (STORE) {
    if (n > 0 && Xfq) {
      const long xb = (((long)s * H + h) * NB + zb) * DK;
      store_state_q(Xfq + xb * BV, Xfs + xb);
    }
  }
  if (ht) store_state(ht + soff);
}

// Boundary states of the segmented forward (run_fwd_bf).  A sequence cut into P
// segments of equal length is P virtual rows s P + p; the state recurrence is
// affine in the state entering a segment, so with Phi_p (dk x dk) the product
// of segment p's chunk transitions and F_p (dk x dv) its final state from a
// zero start, the true states entering the segments are
//   X_0 = h0 (or 0),   X_{p+1} = Phi_p X_p + F_p.
// X_p is written to X0 [row s P + p].  One workgroup per (sequence, head,
// SEG_SL-column slice: many small workgroups, since few rows are cut); the
// slice of X lives in LDS, thread t forms row t / TPR, columns c0 .. c0 + CPT
// - 1 of the next one in fp32 (fixed summation order).
constexpr int SEG_SL = 8;
template <int DK, int DV>
__global__ __launch_bounds__(NTHR) void k_seg_combine(const float* __restrict__ phi,
                                                      const float* __restrict__ F,
                                                      const float* __restrict__ h0, int P, int H,
                                                      float* __restrict__ X0) {
  constexpr int SL = SEG_SL, TPR = NTHR / DK, CPT = SL / TPR;
  static_assert(NTHR % DK == 0 && SL % TPR == 0, "rows per workgroup");
  constexpr int NSL = DV / SL;
  const int zb = blockIdx.x % NSL, sh = blockIdx.x / NSL, h = sh % H, s = sh / H;
  const int j0 = zb * SL;
  const int r = threadIdx.x / TPR, c0 = (threadIdx.x % TPR) * CPT;
  const size_t sdv = (size_t)DK * DV, sdk = (size_t)DK * DK;
  __shared__ float Xs[DK][SL + 1];
  for (int i = threadIdx.x; i < DK * SL; i += NTHR) {
    const int rr = i / SL, cc = i % SL;
    Xs[rr][cc] = h0 ? h0[((size_t)s * H + h) * sdv + (size_t)rr * DV + j0 + cc] : 0.f;
  }
  __syncthreads();
  for (int p = 0; p < P; ++p) {
    const size_t row = ((size_t)s * P + p) * H + h;
    float* x0 = X0 + row * sdv + j0;
    for (int i = threadIdx.x; i < DK * SL; i += NTHR) {
      const int rr = i / SL, cc = i % SL;
      x0[(size_t)rr * DV + cc] = Xs[rr][cc];
    }
    if (p + 1 == P) break;
    const float* ph = phi + row * sdk + (size_t)r * DK;  // row r of Phi_p
    const float* f = F + row * sdv + (size_t)r * DV + j0 + c0;
    float acc[CPT];
#pragma unroll
    for (int j = 0; j < CPT; ++j) acc[j] = f[j];
    for (int kk = 0; kk < DK; ++kk) {
      const float a = ph[kk];
#pragma unroll
      for (int j = 0; j < CPT; ++j) acc[j] = fmaf(a, Xs[kk][c0 + j], acc[j]);
    }
    __syncthreads();  // every row of X_p has been read
#pragma unroll
    for (int j = 0; j < CPT; ++j) Xs[r][c0 + j] = acc[j];
    __syncthreads();
  }
}

// Boundary gradients of the segmented backward.  Y at the end of a row's last
// segment is dht (or 0); the reverse recurrence is affine in it, with the
// transposed transition product Phi_p^T of segment p, so with G_p (dk x dv)
// segment p's state gradient at its start from a zero end (virtual row s P + p
// of both), the gradient of the state leaving segment p - 1 is
//   Y_{p-1} = Phi_p^T Y_p + G_p,   p = P-1 .. 1.
// Y_p goes to Y0 [row s P + p] (the reverse scan's end state of segment p).
// Workgroups as in k_seg_combine.
template <int DK, int DV>
__global__ __launch_bounds__(NTHR) void k_seg_combine_bwd(const float* __restrict__ phi,
                                                          const float* __restrict__ G,
                                                          const float* __restrict__ dht, int P,
                                                          int H, float* __restrict__ Y0) {
  constexpr int SL = SEG_SL, TPR = NTHR / DK, CPT = SL / TPR;
  static_assert(NTHR % DK == 0 && SL % TPR == 0, "rows per workgroup");
  constexpr int NSL = DV / SL;
  const int zb = blockIdx.x % NSL, sh = blockIdx.x / NSL, h = sh % H, s = sh / H;
  const int j0 = zb * SL;
  const int r = threadIdx.x / TPR, c0 = (threadIdx.x % TPR) * CPT;
  const size_t sdv = (size_t)DK * DV, sdk = (size_t)DK * DK;
  __shared__ float Ys[DK][SL + 1];
  for (int i = threadIdx.x; i < DK * SL; i += NTHR) {
    const int rr = i / SL, cc = i % SL;
    Ys[rr][cc] = dht ? dht[((size_t)s * H + h) * sdv + (size_t)rr * DV + j0 + cc] : 0.f;
  }
  __syncthreads();
  for (int p = P - 1; p >= 0; --p) {
    const size_t row = ((size_t)s * P + p) * H + h;
    float* y0 = Y0 + row * sdv + j0;
    for (int i = threadIdx.x; i < DK * SL; i += NTHR) {
      const int rr = i / SL, cc = i % SL;
      y0[(size_t)rr * DV + cc] = Ys[rr][cc];
    }
    if (p == 0) break;
    const float* ph = phi + row * sdk + r;  // column r of Phi_p
    const float* gp = G + row * sdv + (size_t)r * DV + j0 + c0;
    float acc[CPT];
#pragma unroll
    for (int j = 0; j < CPT; ++j) acc[j] = gp[j];
    for (int kk = 0; kk < DK; ++kk) {
      const float a = ph[(size_t)kk * DK];
#pragma unroll
      for (int j = 0; j < CPT; ++j) acc[j] = fmaf(a, Ys[kk][c0 + j], acc[j]);
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < CPT; ++j) Ys[r][c0 + j] = acc[j];
    __syncthreads();
  }
}

// Reverse state scan (bf16 inputs): Y = gradient of the state leaving the chunk.
// As in the forward scan, every product is formed transposed, so that a lane
// holds one row and four consecutive columns; the intermediate tiles (Y, dO,
// dD, Pg, W2) sit row-major in LDS and are read as operands with transposing
// reads.
// STORE = false: the recurrence alone (no Y, dR stores), for the segmented
// backward's state pass.
template <int DK, int DV, int BV, bool STORE = true>
__global__ __launch_bounds__(NTHR, 1) void k_scan_bwd_bf(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ k, const bf16_t* __restrict__ dO,
    const bf16_t* __restrict__ beta_tilde, const float* __restrict__ d, const float* __restrict__ dht,
    const SeqInfo* __restrict__ smap, const int* __restrict__ sorder, int N, int Tfix, int H,
    const int16_t* __restrict__ Mq,
    const float* __restrict__ Ms, const int16_t* __restrict__ Aq, const float* __restrict__ As,
    const bf16_t* __restrict__ QTp,
    const float* __restrict__ Gw, float* __restrict__ dh0, int16_t* __restrict__ Yq,
    float* __restrict__ Ys, int16_t* __restrict__ dRq, float* __restrict__ dRs, int grp = 0,
    int goff = 0) {
  // as in the forward scan, all loop memory operations are unconditional
  constexpr int NTV = BV / 16, XMT = DK / 64, KS = DK / 32, CC = CH * CH;
  constexpr int NB = DV / 32;
  constexpr int LDT = BV + 4;  // row-major BV-wide tiles (see the forward scan)
  static_assert(BV == 32, "stored states use one scale per 32-column block = one dv slice");
  __shared__ __align__(16) bf16_t Yh[DK * LDT];
  __shared__ __align__(16) bf16_t Yl[DK * LDT];
  __shared__ __align__(16) bf16_t dOs[2][CH * LDT];
  __shared__ __align__(16) bf16_t dDh[CH * LDT];
  __shared__ __align__(16) bf16_t dDl[CH * LDT];
  __shared__ __align__(16) bf16_t Pgh[CH * LDT];
  __shared__ __align__(16) bf16_t Pgl[CH * LDT];
  __shared__ __align__(16) bf16_t W2h[CH * LDT];
  __shared__ __align__(16) bf16_t W2l[CH * LDT];

  int s, h, zb;
  if (!scan_item<DV / BV>(N, H, sorder, s, h, zb, grp, goff)) return;
  const int j0 = zb * BV;
  const SeqInfo si = seq_at(smap, s, Tfix);
  const int w = wave_id(), lane = lane_id(), r16 = lane & 15, g4 = lane >> 4;
  const long soff = ((long)s * H + h) * DK * DV;
  const float dh = d[h];
  const int n = si.nchunks;
  const int prow = 16 * w + r16;            // chunk row of this lane
  const int yrow0 = (DK / 4) * w + r16;     // state rows of this lane: yrow0 + 16 mt
  const int col0 = 4 * g4;                  // columns of this lane: 16 nt + col0 .. +3

  floatx4 Y[XMT][NTV];
#pragma unroll
  for (int mt = 0; mt < XMT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NTV; ++nt) {
      if (dht) {
        const float4 y4 = *reinterpret_cast<const float4*>(dht + soff + (long)(yrow0 + 16 * mt) * DV + j0 + 16 * nt + col0);
        Y[mt][nt] = floatx4{y4.x, y4.y, y4.z, y4.w};
      } else {
        Y[mt][nt] = zero4();
      }
    }
  auto put_state = [&]() {
#pragma unroll
    for (int mt = 0; mt < XMT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt) {
        const float yv[4] = {Y[mt][nt][0], Y[mt][nt][1], Y[mt][nt][2], Y[mt][nt][3]};
        put_t4(Yh, Yl, (yrow0 + 16 * mt) * LDT + 16 * nt + col0, yv);
      }
  };
  auto store_state = [&](float* dst) {
#pragma unroll
    for (int mt = 0; mt < XMT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt)
        store4(dst + (long)(yrow0 + 16 * mt) * DV + j0 + 16 * nt + col0, Y[mt][nt]);
  };
  // the same rows as int16 with one scale per row of the slice (see q_pack4),
  // into the slice's own block: dq = block base, [DK][BV]; ds = its row scales
  // (16-byte stores and one scale store, as in the forward scan)
  auto store_state_q = [&](int16_t* dq, float* ds) {
    float sc = 0.f;
#pragma unroll
    for (int mt = 0; mt < XMT; ++mt) {
      float m = nmax_abs4(nmax_abs4(0.f, Y[mt][0]), Y[mt][1]);
      m = rowgroup_max(m);
      const float inv = q_inv_scale(m);
      const unsigned row = yrow0 + 16 * mt;
      at(reinterpret_cast<uint4*>(dq), 2u * (row * BV + row8_col())) =
          row8_from_pieces(q_pack4(Y[mt][0], inv), q_pack4(Y[mt][1], inv));
      if (g4 == mt) sc = q_scale(m);
    }
    if (g4 < XMT) at(ds, 4u * (yrow0 + 16 * g4)) = sc;
  };
  put_state();

  // chunk offsets in scalar registers (see the forward scan)
  auto c_len = [&](int cc) { return min(CH, si.len - cc * CH); };
  auto c_tok = [&](int cc) { return (long)__builtin_amdgcn_readfirstlane(si.tok0 + cc * CH) * H + h; };
  auto c_chh = [&](int cc) { return (long)__builtin_amdgcn_readfirstlane(si.chunk0 + cc) * H + h; };

  // The chunk's K rows, staged from the K operand registers: the state update
  // takes its K operand (reduction down the chunk rows) from here with
  // transposing reads.  Q^T comes from prep in fragment order (staging Q rows
  // like K cost this scan more than the copy saves).
  bf16x8 kf[KS], qtf[XMT][2];
  constexpr int LDKC = DK + 24;  // 304-byte rows: conflict-free transposing reads
  __shared__ __align__(16) bf16_t Kc[CH * LDKC];
  // M and A of the chunk as int16, row-major: each lane stores the 16 bytes it
  // loads in fragment order (8 consecutive columns of one row), and transposing
  // reads return the B operands of M^T dD and A^T dO.  M's row scale is folded
  // into the rows of dD (exact: a power of two), A's column scale taken out of
  // the rows of A^T dO.  A is read at the start of a chunk, so the next
  // chunk's A is staged at the end of the current one; M is staged in the
  // chunk's first phase and read in its second.
  constexpr int LDM = CH + 8;  // 144-byte rows: a transposing read's four rows on disjoint banks
  __shared__ __align__(16) int16_t Mt_s[CH * LDM];
  __shared__ __align__(16) int16_t At_s[CH * LDM];
  uint4 aq[2], mq[2];
  float asc, msc;
  // per-row values (G, beta~) and the dO slice are loaded one chunk ahead into
  // registers and staged through double-buffered LDS at the end of each chunk
  __shared__ float Grow[2][CH], Brow[2][CH];
  float pgv = 0.f;
  bf16_t pbv = 0;
  int plen = 0;
  uint4 pdo = make_uint4(0, 0, 0, 0);  // next chunk's dO slice, 16 bytes per thread
  // rows past the chunk end load a valid row; dD is zeroed there at use
  auto load_k = [&](int cc) {
    const bf16x8* kc = reinterpret_cast<const bf16x8*>(k + c_tok(cc) * DK);
    const unsigned rb = 2u * ((unsigned)min(prow, c_len(cc) - 1) * (H * DK) + 8 * g4);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) kf[ks] = at(kc, rb + 64u * ks);
  };
  const unsigned foff = 16u * (2 * w * 64 + lane);  // this lane's fragment (fragment order)
  // A's fragments and the column scale of A's column prow
  auto load_a = [&](int cc) {
    const uint4* p = reinterpret_cast<const uint4*>(Aq + c_chh(cc) * CC);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) aq[ks] = at(p, foff + 1024u * ks);
    asc = at(As + c_chh(cc) * CH, 4u * prow);
  };
  // M's fragments and the scale of M's row prow
  auto load_m = [&](int cc) {
    const uint4* p = reinterpret_cast<const uint4*>(Mq + c_chh(cc) * CC);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) mq[ks] = at(p, foff + 1024u * ks);
    msc = at(Ms + c_chh(cc) * CH, 4u * prow);
  };
  // fragment (row 16 w + r16, columns 32 ks + 8 g4 ..) to its row-major place
  // (the fragments by value: a reference to the register arrays would keep
  // them in memory)
  auto put_frag = [&](int16_t* t, uint4 r0, uint4 r1) {
    *reinterpret_cast<uint4*>(t + (16 * w + r16) * LDM + 8 * g4) = r0;
    *reinterpret_cast<uint4*>(t + (16 * w + r16) * LDM + 32 + 8 * g4) = r1;
  };
  // lane (g4, r16): column 16 w + r16 of the tile at rows 32 ks + 8 g4 .. +7
  auto get_tr = [&](const int16_t* t, int ks) {
    return __builtin_bit_cast(uint4, ld_tr8(reinterpret_cast<const bf16_t*>(t), LDM, 32 * ks + 8 * g4, 16 * w));
  };
  const unsigned qoff = 16u * (2 * XMT * w * 64 + lane);
  auto load_qt = [&](int cc) {
    // fragment order: rows (DK/4) w + 16 mt + i are row block w XMT + mt
    const bf16x8* p = reinterpret_cast<const bf16x8*>(QTp + c_chh(cc) * DK * CH);
#pragma unroll
    for (int mt = 0; mt < XMT; ++mt)
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) qtf[mt][ks] = at(p, qoff + 1024u * (2 * mt + ks));
  };
  auto load_rows = [&](int cc) {
    plen = c_len(cc);
    const long tok = c_tok(cc), chh = c_chh(cc);
    const int t = threadIdx.x & (CH - 1);
    pgv = at(Gw + chh * CH, 4u * t);
    pbv = at(beta_tilde + tok, 2u * ((unsigned)min(t, plen - 1) * H));
  };
  auto put_rows = [&](int buf) {
    const int t = threadIdx.x & (CH - 1);
    Grow[buf][t] = pgv;
    Brow[buf][t] = t < plen ? bf2f(pbv) : 0.f;
  };
  // dO slice of a chunk: 64 tokens x BV columns in 16-byte pieces; thread t
  // (t < 8 BV) holds token t / (BV/8), columns 8 (t % (BV/8)) .. +7; staged
  // row-major (rows past the chunk end zero)
  constexpr int DPR = BV / 8;
  const int dr = threadIdx.x / DPR, dc = (threadIdx.x % DPR) * 8;
  const bool do_thr = CH * DPR >= NTHR || threadIdx.x < CH * DPR;
  const int dr_ld = min(dr, CH - 1);
  int do_ok = 0;
  auto load_do = [&](int cc) {
    const int len = c_len(cc);
    do_ok = do_thr && dr < len;
    pdo = at(reinterpret_cast<const uint4*>(dO + c_tok(cc) * DV + j0),
             2u * ((unsigned)min(dr_ld, len - 1) * (H * DV) + dc));
  };
  auto put_do = [&](int buf) {
    const uint4 val = do_ok ? pdo : make_uint4(0, 0, 0, 0);
    if (do_thr) {
      // two 8-byte writes: the 72-byte rows keep only 8-byte alignment
      *reinterpret_cast<uint2*>(dOs[buf] + dr * LDT + dc) = make_uint2(val.x, val.y);
      *reinterpret_cast<uint2*>(dOs[buf] + dr * LDT + dc + 4) = make_uint2(val.z, val.w);
    }
  };

  if (n > 0) {
    load_do(n - 1);
    load_k(n - 1);
    load_a(n - 1);
    load_m(n - 1);
    load_qt(n - 1);
    load_rows(n - 1);
    put_rows((n - 1) & 1);
    put_do((n - 1) & 1);
    put_frag(At_s, aq[0], aq[1]);  // the loop stages each next chunk's A
  }
  __syncthreads();

  for (int cc = n - 1; cc >= 0; --cc) {
    const bool more = cc > 0;
    const int nx = more ? cc - 1 : cc;  // chunk prefetched during this one
    const long chh = c_chh(cc);
    const int buf = cc & 1;
    const int clen = c_len(cc);
    load_rows(nx);
    load_do(nx);
    const float glast = Grow[buf][CH - 1];
    // G_{r-1} read unconditionally (row 0 reads G_0 and drops it): a read
    // under the row-0 branch waited for the LDS on the spot every chunk (-1.7%
    // here; in the forward scan the same change measured +2.7% and is not made)
    const float gp = Grow[buf][max(prow - 1, 0)];
    const float gg = Grow[buf][prow], gm = prow > 0 ? gp : 0.f, bb = Brow[buf][prow];

    // dD = A^T dO + Diag(exp(G_63 - G)) K Y, formed transposed
    floatx4 ky[NTV], ad[NTV];
#pragma unroll
    for (int nt = 0; nt < NTV; ++nt) {
      ky[nt] = zero4();
      ad[nt] = zero4();
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt) {
        const bf16x8 yh = ld_tr8(Yh, LDT, 32 * ks + 8 * g4, 16 * nt);
        const bf16x8 yl = ld_tr8(Yl, LDT, 32 * ks + 8 * g4, 16 * nt);
        ky[nt] = mfma16(yh, kf[ks], ky[nt]);
        ky[nt] = mfma16(yl, kf[ks], ky[nt]);
      }
    // the state gradient of this chunk, stored while the products run (stores
    // bunched before a barrier stall all four waves at once)
    if constexpr (STORE) store_state_q(Yq + (chh * NB + zb) * DK * BV, Ys + (chh * NB + zb) * DK);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      bf16x8 ath, atl;
      q_split8(get_tr(At_s, ks), ath, atl);
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt) {
        const bf16x8 dov = ld_tr8(dOs[buf], LDT, 32 * ks + 8 * g4, 16 * nt);
        ad[nt] = mfma16(dov, ath, ad[nt]);
        ad[nt] = mfma16(dov, atl, ad[nt]);
      }
    }
    const float at_cur = asc;
    // K rows past the chunk end repeat row len - 1; W2 is zero there
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) *reinterpret_cast<bf16x8*>(Kc + prow * LDKC + 32 * ks + 8 * g4) = kf[ks];
    put_frag(Mt_s, mq[0], mq[1]);
    load_k(nx);
    load_a(nx);
    {
      // dD rows times M's row scale (the reduction index of M^T dD)
      const float edec = prow < clen ? __expf(glast - gg) * msc : 0.f,
                  atm = prow < clen ? at_cur * msc : 0.f;
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt) {
        float dd_[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) dd_[e] = atm * ad[nt][e] + edec * ky[nt][e];
        put_t4(dDh, dDl, prow * LDT + 16 * nt + col0, dd_);
      }
    }
    __syncthreads();

    // dR = M^T dD;  Pg = Diag(exp G) dO;  W2 = -d Pg - Diag(beta~ exp Gm) dR
    floatx4 drr[NTV];
#pragma unroll
    for (int nt = 0; nt < NTV; ++nt) drr[nt] = zero4();
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      bf16x8 mth, mtl;
      q_split8(get_tr(Mt_s, ks), mth, mtl);
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt) {
        const bf16x8 xh = ld_tr8(dDh, LDT, 32 * ks + 8 * g4, 16 * nt);
        const bf16x8 xl = ld_tr8(dDl, LDT, 32 * ks + 8 * g4, 16 * nt);
        drr[nt] = mfma16(xh, mth, drr[nt]);
        drr[nt] = mfma16(xl, mth, drr[nt]);
        drr[nt] = mfma16(xh, mtl, drr[nt]);
      }
    }
    load_m(nx);
    // the K fragments of the state update (state rows (dk/4) w + 16 mt + r16,
    // chunk rows 32 ks + 8 g4 ..): the tile is complete since the first
    // barrier, so they are read here, off the update's path
    bf16x8 ktf[2][XMT];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int mt = 0; mt < XMT; ++mt) ktf[ks][mt] = ld_tr8(Kc, LDKC, 32 * ks + 8 * g4, (DK / 4) * w + 16 * mt);
    // dR rows as int16 with one scale per row of the slice, stored after the
    // next phase's products are issued
    uint4 rpk;
    float rsc;
    {
      const float m = rowgroup_max(nmax_abs4(nmax_abs4(0.f, drr[0]), drr[1]));
      const float inv = q_inv_scale(m);
      rpk = row8_from_pieces(q_pack4(drr[0], inv), q_pack4(drr[1], inv));
      rsc = q_scale(m);
    }
    {
      const float eg = __expf(gg), begm = bb * __expf(gm);
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt) {
        const int off = prow * LDT + 16 * nt + col0;
        const uint2 d4 = *reinterpret_cast<const uint2*>(dOs[buf] + off);
        const float dov[4] = {__uint_as_float(d4.x << 16), __uint_as_float(d4.x & 0xFFFF0000u),
                              __uint_as_float(d4.y << 16), __uint_as_float(d4.y & 0xFFFF0000u)};
        float pg[4], w2[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          pg[e] = eg * dov[e];
          w2[e] = -dh * pg[e] - begm * drr[nt][e];
        }
        put_t4(Pgh, Pgl, off, pg);
        put_t4(W2h, W2l, off, w2);
      }
    }
    __syncthreads();

    // Y^T <- exp(G_63) Y^T + Pg^T Q + W2^T K
    const float gC = __expf(glast);
#pragma unroll
    for (int mt = 0; mt < XMT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt) Y[mt][nt] *= gC;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
      for (int nt = 0; nt < NTV; ++nt) {
        const bf16x8 ph = ld_tr8(Pgh, LDT, 32 * ks + 8 * g4, 16 * nt);
        const bf16x8 pl = ld_tr8(Pgl, LDT, 32 * ks + 8 * g4, 16 * nt);
        const bf16x8 wh = ld_tr8(W2h, LDT, 32 * ks + 8 * g4, 16 * nt);
        const bf16x8 wl = ld_tr8(W2l, LDT, 32 * ks + 8 * g4, 16 * nt);
#pragma unroll
        for (int mt = 0; mt < XMT; ++mt) {
          Y[mt][nt] = mfma16(ph, qtf[mt][ks], Y[mt][nt]);
          Y[mt][nt] = mfma16(pl, qtf[mt][ks], Y[mt][nt]);
          Y[mt][nt] = mfma16(wh, ktf[ks][mt], Y[mt][nt]);
          Y[mt][nt] = mfma16(wl, ktf[ks][mt], Y[mt][nt]);
        }
      }
    }
    if constexpr (STORE) {
      const long blk = (chh * NB + zb) * CH;  // the slice's block
      at(reinterpret_cast<uint4*>(dRq + blk * BV), 2u * (prow * BV + row8_col())) = rpk;
      if (g4 == 0) at(dRs + blk, 4u * prow) = rsc;
    }
    load_qt(nx);
    // the next chunk's A (this chunk's was read before the first barrier)
    put_frag(At_s, aq[0], aq[1]);
    put_do(buf ^ 1);
    put_rows(buf ^ 1);
    put_state();
    __syncthreads();
  }
  if (dh0) store_state(dh0 + soff);
}

// ---------------------------------------------------------------------------
// k_intra_bwd_bf: per chunk-head gradients for bf16 inputs, 8 wavefronts.
// Wave w works on row tile rt = w % 4 (rows 16 rt .. 16 rt + 15) and column
// half ch = w / 4 of every chunk product.  Phase 1 streams dv in blocks of 32
// (prefetched one block ahead; the int16 operands are dequantised and split
// into bf16 hi/lo once, when staged into LDS) and accumulates T1 = dO X^T,
// T3 = dR X^T, T2 = D Y^T, dA = dO D^T, dL = dR D^T.  The K and Q tiles are
// loaded with the first block into LDS of their own; phase 2 forms dQ~ and dK
// from them (K^T, Q^T B-operands by transposing LDS reads).
// ---------------------------------------------------------------------------
constexpr int IB_THR = 512;

template <int DK>
struct IntraBwdBfSmem {
  static constexpr int VB = 32, LDB = VB + 8;
  static constexpr int LDK = DK + 24, LDC = CH + 8;  // K, Q: conflict-free 16-byte and transposing reads
  static constexpr int P1 = (6 * CH * LDB + 4 * DK * LDB) * 2;
  static constexpr int P2 = (2 * CH * LDK + 6 * CH * LDC) * 2;
  static constexpr int BYTES = P1 > P2 ? P1 : P2;
};

__device__ __forceinline__ void split4v(const float4& x, bf16x4& hi, bf16x4& lo) {
  const float a[4] = {x.x, x.y, x.z, x.w};
  split4(a, hi, lo);
}

// Per-row values of a lane's four accumulator rows r0 .. r0 + 3 (r0 % 4 == 0,
// Gs and Bts 16-byte aligned): G_r, G_{r-1} (G_0 stands in at r = 0, where
// no term uses it) and beta~_r.
struct RowVals {
  float g[4], gm[4], bt[4];
};
__device__ __forceinline__ RowVals row_vals(const float* Gs, const float* Bts, int r0) {
  const float4 g = *reinterpret_cast<const float4*>(Gs + r0);
  const float4 b = *reinterpret_cast<const float4*>(Bts + r0);
  const float gp = Gs[max(r0 - 1, 0)];
  return RowVals{{g.x, g.y, g.z, g.w}, {gp, g.x, g.y, g.z}, {b.x, b.y, b.z, b.w}};
}

// The gate terms of entry (r, c) of the chunk's 64 x 64 gradient products:
// gam = e^{G_r - G_c} on and below the diagonal, lc = e^{G_{r-1} - G_c} below
// it.  Branch-free: both exponentials are evaluated for every entry and the
// masked values are selected away (above the diagonal they may overflow).
struct GateTerms {
  float e1, e2, dag, dakk;
};
__device__ __forceinline__ GateTerms gate_terms(int r, int c, const RowVals& rv, int e, float Gc,
                                                float kk, float qk, float da, float dLv, float dh,
                                                float& rbl) {
  const bool on = r >= c, below = r > c;
  const float gam = __expf(rv.g[e] - Gc), lc = __expf(rv.gm[e] - Gc);
  const float a = (qk - dh * kk) * gam;
  const float dl = -dLv;
  const float lck = lc * kk;
  rbl = below ? rbl + dl * lck : rbl;
  GateTerms t;
  t.e1 = on ? da * a : 0.f;
  t.dag = on ? da * gam : 0.f;
  t.e2 = below ? dl * rv.bt[e] * lck : 0.f;
  t.dakk = below ? dl * rv.bt[e] * lc : 0.f;
  return t;
}

template <int DK, int DV>
__global__ __launch_bounds__(IB_THR, 1) void k_intra_bwd_bf(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ k, const bf16_t* __restrict__ v,
    const bf16_t* __restrict__ dO, const bf16_t* __restrict__ beta,
    const bf16_t* __restrict__ beta_tilde, const float* __restrict__ d,
    const ChunkInfo* __restrict__ cmap, int Tfix, int H, const float* __restrict__ Gw,
    const int16_t* __restrict__ Xq, const float* __restrict__ Xs, const int16_t* __restrict__ Dq,
    const float* __restrict__ Ds, const int16_t* __restrict__ Yq, const float* __restrict__ Ys,
    const int16_t* __restrict__ dRq, const float* __restrict__ dRs, int ncmax, float* __restrict__ dq, float* __restrict__ dk,
    float* __restrict__ dv, float* __restrict__ dbeta, float* __restrict__ dbeta_tilde,
    float* __restrict__ dg, float* __restrict__ ddp) {
  using SM = IntraBwdBfSmem<DK>;
  constexpr int VB = SM::VB, LDB = SM::LDB, LDK = SM::LDK, LDC = SM::LDC;
  constexpr int NTW = DK / 32;          // dk column tiles per wave
  constexpr int NW = IB_THR / 64;       // wavefronts
  constexpr int NVB = DV / VB;
  constexpr int XP = DK * (VB / 4) / IB_THR;  // X / Y 16-byte pieces per thread
  __shared__ __align__(16) char smem[SM::BYTES];
  // Bs: beta (write strength: dv), Bts: beta~ (feedback strength: L and R's
  // K X term); rowB: <v, dR> per row, the derivative through beta
  __shared__ __align__(16) float Gs[CH], Bs[CH], Bts[CH], rowB[CH];
  __shared__ float colpart[4][CH];      // per row tile: column sums of E1 + E2
  __shared__ float rowacc[2][6][CH];    // per column half: E1, E2, BL, p1, p2, p3 row sums
  __shared__ float scal[NW][2];         // per wave: <X, Y>_F, sum k . dQ~
  // The next item's first phase-1 block, copied from memory straight into LDS
  // while this item is in phase 2 (which loads nothing else): the X, Y, dR, D
  // blocks as stored, the dO and v rows of the first block pair, their scales.
  // Every region is a whole number of 1 KiB pieces, one wave-wide 16-byte copy
  // each.
  constexpr int RX = 64 * DK, RD = 64 * CH, RP = 128 * CH;  // bytes: X or Y, dR or D, dO or v pair
  constexpr int O_Y = RX, O_DR = 2 * RX, O_D = O_DR + RD, O_DO = O_D + RD, O_V = O_DO + RP;
  constexpr int O_XS = O_V + RP, O_RS = O_XS + 1024, RAW = O_RS + 1024;
  static_assert(RX % 1024 == 0 && RD % 1024 == 0 && 8 * DK <= 1024 && 8 * CH <= 1024, "1 KiB pieces");
  static_assert(2 * (RX / 1024) % NW == 0 && 2 * (RD / 1024) == NW && RP / 1024 == NW,
                "the copies take whole rounds of one piece per wave");
  __shared__ __align__(16) char R0[RAW];

  // Persistent: workgroup b takes items b, b + gridDim.x, ... (item = chunk +
  // ncmax * head).
  const int nitems = ncmax * H;
  bool have = false;            // the item's first block is waiting in R0
  float g_nx = 0.f;              // and its gates
  bf16_t b_nx = 0, bt_nx = 0;    // and beta, beta~ (raw: converted only when the item starts)
  for (int item = blockIdx.x; item < nitems; item += gridDim.x) {
  // The thread index passes through an opaque copy every item, so that the
  // values derived from it are formed inside the loop instead of being held
  // in registers across it.
  int tid;
  asm volatile("v_mov_b32 %0, %1" : "=v"(tid) : "v"((int)threadIdx.x));
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63, r16 = lane & 15, g4 = lane >> 4;
  const int rt = w & 3, ch = w >> 2;
  const int h = item / ncmax;
  const long chh = (long)(item % ncmax) * H + h;
  const ChunkInfo ci = chunk_at(cmap, item % ncmax, Tfix);
  if (ci.len <= 0) {
    if (tid == 0) ddp[chh] = 0.f;
    have = false;
    continue;
  }
  const long tok = (long)ci.tok0 * H + h;
  const int len = ci.len;
  const float dh = d[h];

  // ---------------- phase 1 ----------------
  bf16_t* dOb = reinterpret_cast<bf16_t*>(smem);
  bf16_t* dRh = dOb + CH * LDB;
  bf16_t* dRl = dRh + CH * LDB;
  bf16_t* Dh = dRl + CH * LDB;
  bf16_t* Dl = Dh + CH * LDB;
  bf16_t* Xh = Dl + CH * LDB;
  bf16_t* Xl = Xh + DK * LDB;
  bf16_t* Yh = Xl + DK * LDB;
  bf16_t* Yl = Yh + DK * LDB;
  bf16_t* Vb = Yl + DK * LDB;

  // dO and v arrive two blocks at a time, whole 128-byte lines: thread t holds
  // row t / 8, columns 8 (t % 8) .. +7 of the 64 columns of blocks (2p, 2p+1),
  // i.e. a piece of block 2p + pb; it stages the piece when that block comes up
  const int pr = tid >> 3, pc = (tid & 7) * 8, pb = (tid & 7) >> 2;
  const int pf_r = tid >> 3, pf_c = (tid & 7) * 4;                 // dR / D piece
  // X, Y, D, dR arrive as int16 with one scale per (row, 32-column block), each
  // 32-column block stored on its own ([chunk-head][block][row][32]): the block
  // is exactly one VB-wide phase-1 step (see q_pack4)
  static_assert(VB == 32, "column blocks must match the stored scale blocks");
  constexpr int NB = DV / 32;
  uint4 r_do, r_v;
  uint2 r_dr, r_d, r_x[XP], r_y[XP];
  float s_dr, s_d, s_x[XP], s_y[XP];
  static_assert(NVB % 2 == 0 && CH * 8 == IB_THR, "dO / v pairs: one 16-byte piece per thread");
  // this chunk-head's operands: scalar bases, 32-bit per-lane byte offsets
  const bf16_t* dO_i = dO + tok * DV;  // row r at r H DV
  const bf16_t* v_i = v + tok * DV;
  const int16_t* dRq_i = dRq + chh * NB * CH * VB;  // [block][row][32]
  const int16_t* Dq_i = Dq + chh * NB * CH * VB;
  const float* dRs_i = dRs + chh * NB * CH;         // [block][row]
  const float* Ds_i = Ds + chh * NB * CH;
  const int16_t* Xq_i = Xq + chh * NB * DK * VB;
  const int16_t* Yq_i = Yq + chh * NB * DK * VB;
  const float* Xs_i = Xs + chh * NB * DK;
  const float* Ys_i = Ys + chh * NB * DK;
  auto issue = [&](int vb) {
    if (vb % 2 == 0) {
      const unsigned rb = 2u * ((unsigned)min(pr, len - 1) * (H * DV) + vb * VB + pc);
      r_do = at(reinterpret_cast<const uint4*>(dO_i), rb);
      r_v = at(reinterpret_cast<const uint4*>(v_i), rb);
    }
    const unsigned rr = vb * CH + pf_r;
    r_dr = at(reinterpret_cast<const uint2*>(dRq_i), 2u * (rr * VB + pf_c));
    r_d = at(reinterpret_cast<const uint2*>(Dq_i), 2u * (rr * VB + pf_c));
    s_dr = at(dRs_i, 4u * rr);
    s_d = at(Ds_i, 4u * rr);
#pragma unroll
    for (int p = 0; p < XP; ++p) {
      const int pc = tid + p * IB_THR, xr = pc >> 3, xc = (pc & 7) * 4;
      const unsigned xrow = vb * DK + xr;
      r_x[p] = at(reinterpret_cast<const uint2*>(Xq_i), 2u * (xrow * VB + xc));
      r_y[p] = at(reinterpret_cast<const uint2*>(Yq_i), 2u * (xrow * VB + xc));
      s_x[p] = at(Xs_i, 4u * xrow);
      s_y[p] = at(Ys_i, 4u * xrow);
    }
    // keep the loads here: the scheduler otherwise sinks some of them to their
    // use one block later, where they are waited for at once
    __builtin_amdgcn_sched_barrier(0);
  };
  float Fpart = 0.f, bv = 0.f;
  float4 fdr;  // this thread's dR piece, kept for <v_r, dR_r> after the barrier
  // this chunk's dv rows (row r at r H DV), bounded at row len
  const __amdgpu_buffer_rsrc_t rdv = clip_rsrc(dv + tok * DV, (unsigned)len * (unsigned)(H * DV * 4));
  auto put = [&](int vb) {
    const int j = vb * VB;
    if (pb == (vb & 1)) {
      *reinterpret_cast<uint4*>(dOb + pr * LDB + (pc & 31)) = r_do;
      *reinterpret_cast<uint4*>(Vb + pr * LDB + (pc & 31)) = r_v;
    }
    bf16x4 hh, ll;
    fdr = q_unpack4(r_dr, s_dr);
    split4v(fdr, hh, ll);
    *reinterpret_cast<bf16x4*>(dRh + pf_r * LDB + pf_c) = hh;
    *reinterpret_cast<bf16x4*>(dRl + pf_r * LDB + pf_c) = ll;
    split4v(q_unpack4(r_d, s_d), hh, ll);
    *reinterpret_cast<bf16x4*>(Dh + pf_r * LDB + pf_c) = hh;
    *reinterpret_cast<bf16x4*>(Dl + pf_r * LDB + pf_c) = ll;
#pragma unroll
    for (int p = 0; p < XP; ++p) {
      const int pc = tid + p * IB_THR, xr = pc >> 3, xc = (pc & 7) * 4;
      const float4 fx = q_unpack4(r_x[p], s_x[p]), fy = q_unpack4(r_y[p], s_y[p]);
      split4v(fx, hh, ll);
      *reinterpret_cast<bf16x4*>(Xh + xr * LDB + xc) = hh;
      *reinterpret_cast<bf16x4*>(Xl + xr * LDB + xc) = ll;
      split4v(fy, hh, ll);
      *reinterpret_cast<bf16x4*>(Yh + xr * LDB + xc) = hh;
      *reinterpret_cast<bf16x4*>(Yl + xr * LDB + xc) = ll;
      Fpart += fx.x * fy.x + fx.y * fy.y + fx.z * fy.z + fx.w * fy.w;
    }
    // dv = Diag(beta) dR
    const float b = Bs[pf_r];
    store_clip4(floatx4{b * fdr.x, b * fdr.y, b * fdr.z, b * fdr.w}, rdv,
                4u * ((unsigned)pf_r * (H * DV) + j + pf_c));  // rows >= len dropped
  };

  floatx4 T1[NTW], T2[NTW], T3[NTW], dA[2], dL[2];
#pragma unroll
  for (int j = 0; j < NTW; ++j) {
    T1[j] = zero4();
    T2[j] = zero4();
    T3[j] = zero4();
  }
  dA[0] = dA[1] = dL[0] = dL[1] = zero4();
  TileRegs<bf16_t, CH, DK, IB_THR> kr, qr;
  float g_in, b_in, bt_in;
  if (have) {
    // the copies into R0 were issued by this thread's wave; after the wait
    // and the barrier every wave's copies are in place
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    r_do = *reinterpret_cast<const uint4*>(R0 + O_DO + pr * 128 + pc * 2);
    r_v = *reinterpret_cast<const uint4*>(R0 + O_V + pr * 128 + pc * 2);
    r_dr = *reinterpret_cast<const uint2*>(R0 + O_DR + pf_r * 64 + pf_c * 2);
    r_d = *reinterpret_cast<const uint2*>(R0 + O_D + pf_r * 64 + pf_c * 2);
    s_dr = *reinterpret_cast<const float*>(R0 + O_RS + 4 * pf_r);
    s_d = *reinterpret_cast<const float*>(R0 + O_RS + 4 * CH + 4 * pf_r);
#pragma unroll
    for (int p = 0; p < XP; ++p) {
      const int pc2 = tid + p * IB_THR, xr = pc2 >> 3, xc = (pc2 & 7) * 4;
      r_x[p] = *reinterpret_cast<const uint2*>(R0 + xr * 64 + xc * 2);
      r_y[p] = *reinterpret_cast<const uint2*>(R0 + O_Y + xr * 64 + xc * 2);
      s_x[p] = *reinterpret_cast<const float*>(R0 + O_XS + 4 * xr);
      s_y[p] = *reinterpret_cast<const float*>(R0 + O_XS + 4 * DK + 4 * xr);
    }
    g_in = g_nx;
    b_in = bf2f(b_nx);
    bt_in = bf2f(bt_nx);
  } else {
    issue(0);
    // gates and beta after the first block's loads, unconditional (clamped rows)
    g_in = Gw[chh * CH + (tid & (CH - 1))];
    b_in = bf2f(beta[tok + (long)min(tid & (CH - 1), len - 1) * H]);
    bt_in = bf2f(beta_tilde[tok + (long)min(tid & (CH - 1), len - 1) * H]);
  }
  // unrolled: a rolled loop carries the prefetched registers through copies at
  // the back edge, which wait for the loads just issued
#pragma unroll
  for (int vb = 0; vb < NVB; ++vb) {
    // the scheduler would hoist put's dequantisation across the barrier into
    // the previous block's MFMAs, waiting there for the loads just issued
    __builtin_amdgcn_sched_barrier(0);
    if (vb == 0 && tid < CH) {
      Gs[tid] = g_in;
      Bs[tid] = tid < len ? b_in : 0.f;
      Bts[tid] = tid < len ? bt_in : 0.f;
    }
    __syncthreads();
    put(vb);
    __syncthreads();
    if (vb + 1 < NVB) {
      issue(vb + 1);
    } else {
      kr.load_clip(k + tok * DK, (long)H * DK, len);
      qr.load_clip(q + tok * DK, (long)H * DK, len);
    }
    {
      // <v_r, dR_r> for this thread's piece (v staged by the piece's owner)
      const bf16x4 vv = *reinterpret_cast<const bf16x4*>(Vb + pf_r * LDB + pf_c);
      bv += (float)vv[0] * fdr.x + (float)vv[1] * fdr.y + (float)vv[2] * fdr.z + (float)vv[3] * fdr.w;
    }
    const int arow = (16 * rt + r16) * LDB + 8 * g4;
    // dO rows past the chunk end hold row len - 1 (clamped loads): zero them
    // here, where dO is an MFMA A operand, not on the load's path
    bf16x8 a_do = ld8(dOb + arow);
    if (16 * rt + r16 >= len) a_do = bf16x8{};
    const bf16x8 a_drh = ld8(dRh + arow), a_drl = ld8(dRl + arow);
    const bf16x8 a_dh = ld8(Dh + arow), a_dl = ld8(Dl + arow);
#pragma unroll
    for (int j = 0; j < NTW; ++j) {
      const int brow = (16 * (ch * NTW + j) + r16) * LDB + 8 * g4;
      const bf16x8 xh = ld8(Xh + brow), xl = ld8(Xl + brow);
      const bf16x8 yh = ld8(Yh + brow), yl = ld8(Yl + brow);
      T1[j] = mfma16(a_do, xh, T1[j]);
      T1[j] = mfma16(a_do, xl, T1[j]);
      T3[j] = mfma16(a_drh, xh, T3[j]);
      T3[j] = mfma16(a_drh, xl, T3[j]);
      T3[j] = mfma16(a_drl, xh, T3[j]);
      T2[j] = mfma16(a_dh, yh, T2[j]);
      T2[j] = mfma16(a_dh, yl, T2[j]);
      T2[j] = mfma16(a_dl, yh, T2[j]);
    }
#pragma unroll
    for (int j2 = 0; j2 < 2; ++j2) {
      const int brow = (16 * (2 * ch + j2) + r16) * LDB + 8 * g4;
      const bf16x8 bh = ld8(Dh + brow), bl = ld8(Dl + brow);
      dA[j2] = mfma16(a_do, bh, dA[j2]);
      dA[j2] = mfma16(a_do, bl, dA[j2]);
      dL[j2] = mfma16(a_drh, bh, dL[j2]);
      dL[j2] = mfma16(a_drh, bl, dL[j2]);
      dL[j2] = mfma16(a_drl, bh, dL[j2]);
    }
  }
  bv = sum8(bv);
  if ((tid & 7) == 0) rowB[pf_r] = bv;
  Fpart = wave_sum(Fpart);
  if (lane == 0) scal[w][0] = Fpart;
  __syncthreads();

  // ---------------- phase 2 ----------------
  bf16_t* Ks = reinterpret_cast<bf16_t*>(smem);
  bf16_t* Qs = Ks + CH * LDK;
  // The 64 x 64 gate-term matrices, each (hi, lo), stored in the orientation in
  // which a lane's four accumulator values (rows r .. r+3 of one column c) are
  // contiguous, i.e. at [c][r]; the row-major operands are read back with
  // transposing LDS reads.  With G = dA o Gamma (lower incl. diagonal),
  // P = dAkk (strictly lower) and U = P^T - d G^T (upper incl. diagonal):
  //   GT[c][r] = G[r][c],  PT[c][r] = P[r][c],  Ub[c][r] = U[c][r].
  bf16_t* GTh = Qs + CH * LDK;
  bf16_t* GTl = GTh + CH * LDC;
  bf16_t* PTh = GTl + CH * LDC;
  bf16_t* PTl = PTh + CH * LDC;
  bf16_t* Ubh = PTl + CH * LDC;
  bf16_t* Ubl = Ubh + CH * LDC;
  kr.store(Ks, LDK);
  qr.store(Qs, LDK);
  // Phase 2 reads nothing else from memory: copy the next item's first block
  // into R0 now (one wave-wide 16-byte copy per 1 KiB piece; rows past a chunk
  // end repeat its last row).  The copies are invisible to the compiler's
  // memory-counter bookkeeping: the next item waits for them explicitly.
  {
    const int nx = item + gridDim.x, nxc = min(nx, nitems - 1);
    const ChunkInfo ci2 = chunk_at(cmap, nxc % ncmax, Tfix);
    const int h2 = nxc / ncmax, len2 = ci2.len;
    const long chh2 = (long)(nxc % ncmax) * H + h2, tok2 = (long)ci2.tok0 * H + h2;
    have = nx < nitems && len2 > 0;
    if (have) {
      // Straight-line rounds of one 1 KiB piece per wave: every wave would
      // otherwise run the same per-piece selection on the CU's one scalar unit.
      const unsigned r0 = (unsigned)(size_t)(__attribute__((address_space(3))) void*)R0;
      auto copy = [&](int off, const char* src) {
        // M0 carries the LDS address; the instruction takes it at issue, and
        // the previous M0 is restored (the compiler does not track M0 here)
        const unsigned m0 = __builtin_amdgcn_readfirstlane(r0 + off);
        unsigned m0_saved;
        asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\ts_nop 0\n\t"
                     "global_load_lds_dwordx4 %1, off\n\ts_mov_b32 m0, %0"
                     : "=&s"(m0_saved) : "v"(src), "s"(m0) : "memory");
      };
      const char* xb = reinterpret_cast<const char*>(Xq + chh2 * NB * DK * VB);
      const char* yb = reinterpret_cast<const char*>(Yq + chh2 * NB * DK * VB);
      const char* rb = reinterpret_cast<const char*>(dRq + chh2 * NB * CH * VB);
      const char* db = reinterpret_cast<const char*>(Dq + chh2 * NB * CH * VB);
      // X then Y blocks (RX / 1024 pieces each)
#pragma unroll
      for (int i = 0; i < 2 * (RX / 1024) / NW; ++i) {
        const int j = i * NW + w;
        const char* src = j < RX / 1024 ? xb + 1024 * j : yb + 1024 * (j - RX / 1024);
        copy(1024 * j, src + 16 * lane);
      }
      // dR then D blocks, one round
      {
        const char* src = w < RD / 1024 ? rb + 1024 * w : db + 1024 * (w - RD / 1024);
        copy(O_DR + 1024 * w, src + 16 * lane);
      }
      // dO and v rows of the first block pair, 8 rows per piece (rows past the
      // chunk end repeat its last row)
      {
        const long row = min(8 * w + (lane >> 3), len2 - 1);
        const long e = (tok2 + row * H) * DV + 8 * (lane & 7);
        copy(O_DO + 1024 * w, reinterpret_cast<const char*>(dO + e));
        copy(O_V + 1024 * w, reinterpret_cast<const char*>(v + e));
      }
      if (w == 0) {
        // X then Y scales of block 0 (DK floats each); the rest repeats
        const int l = lane < DK / 2 ? lane : lane & (DK / 4 - 1);
        copy(O_XS, l < DK / 4 ? reinterpret_cast<const char*>(Xs + chh2 * NB * DK) + 16 * l
                              : reinterpret_cast<const char*>(Ys + chh2 * NB * DK) + 16 * (l - DK / 4));
      } else if (w == 1) {
        // dR then D scales of block 0 (CH floats each); the rest repeats
        const int l = lane < CH / 2 ? lane : lane & (CH / 4 - 1);
        copy(O_RS, l < CH / 4 ? reinterpret_cast<const char*>(dRs + chh2 * NB * CH) + 16 * l
                              : reinterpret_cast<const char*>(Ds + chh2 * NB * CH) + 16 * (l - CH / 4));
      }
    }
  }
  __syncthreads();
  const float Glast = Gs[CH - 1];
  // this lane's accumulator rows r0 .. r0 + 3: G_r, G_{r-1} (r > 0) and beta~_r,
  // read once (per-entry reads under the triangle's branches each waited for LDS)
  const RowVals rv = row_vals(Gs, Bts, 16 * rt + 4 * g4);
  {
    floatx4 akk[2], aqk[2];
    akk[0] = akk[1] = aqk[0] = aqk[1] = zero4();
#pragma unroll
    for (int ks = 0; ks < DK / 32; ++ks) {
      const int ar = (16 * rt + r16) * LDK + 32 * ks + 8 * g4;
      const bf16x8 a_k = ld8(Ks + ar), a_q = ld8(Qs + ar);
#pragma unroll
      for (int j2 = 0; j2 < 2; ++j2) {
        const bf16x8 b = ld8(Ks + (16 * (2 * ch + j2) + r16) * LDK + 32 * ks + 8 * g4);
        akk[j2] = mfma16(a_k, b, akk[j2]);
        aqk[j2] = mfma16(a_q, b, aqk[j2]);
      }
    }
    float rE1[4] = {0.f, 0.f, 0.f, 0.f}, rE2[4] = {0.f, 0.f, 0.f, 0.f}, rBL[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j2 = 0; j2 < 2; ++j2) {
      const int c = 16 * (2 * ch + j2) + r16;
      const float Gc = Gs[c];
      float cE = 0.f, dagv[4], pv[4], uv[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const GateTerms t = gate_terms(16 * rt + 4 * g4 + e, c, rv, e, Gc, akk[j2][e], aqk[j2][e],
                                       dA[j2][e], dL[j2][e], dh, rBL[e]);
        dagv[e] = t.dag;
        pv[e] = t.dakk;
        uv[e] = t.dakk - dh * t.dag;  // zero above the diagonal like the others
        rE1[e] += t.e1;
        rE2[e] += t.e2;
        cE += t.e1 + t.e2;
      }
      const int toff = c * LDC + 16 * rt + 4 * g4;
      put_t4(GTh, GTl, toff, dagv);
      put_t4(PTh, PTl, toff, pv);
      put_t4(Ubh, Ubl, toff, uv);
      cE = sum_groups(cE);
      if (g4 == 0) colpart[rt][c] = cE;
    }
    // row dot products of T1, T2, T3 with q~ and k over this wave's columns
    float p1[4] = {0.f, 0.f, 0.f, 0.f}, p2[4] = {0.f, 0.f, 0.f, 0.f}, p3[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < NTW; ++j) {
      // K, Q at this lane's accumulator rows 16 rt + 4 g4 + e of column
      // 16 (ch NTW + j) + r16: one transposing read each
      const bf16x4_t k4 = ld_tr4(Ks, LDK, 16 * rt + 4 * g4, 16 * (ch * NTW + j));
      const bf16x4_t q4 = ld_tr4(Qs, LDK, 16 * rt + 4 * g4, 16 * (ch * NTW + j));
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float kv = (float)k4[e];
        const float qv = (float)q4[e] - dh * kv;
        p1[e] += T1[j][e] * qv;
        p2[e] += T2[j][e] * kv;
        p3[e] += T3[j][e] * kv;
      }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float s0 = sum16(rE1[e]), s1 = sum16(rE2[e]), s2 = sum16(rBL[e]);
      const float s3 = sum16(p1[e]), s4 = sum16(p2[e]), s5 = sum16(p3[e]);
      if (r16 == 0) {
        const int r = 16 * rt + 4 * g4 + e;
        rowacc[ch][0][r] = s0;
        rowacc[ch][1][r] = s1;
        rowacc[ch][2][r] = s2;
        rowacc[ch][3][r] = s3;
        rowacc[ch][4][r] = s4;
        rowacc[ch][5][r] = s5;
      }
    }
  }
  __syncthreads();

  if (w == 0) {
    // Per-row gradients dg, dbeta (lane = row) from the row and column sums:
    // LDS reads only, so this wave forms them ahead of its dQ~, dK products
    // while the other wave on its SIMD keeps the matrix unit busy.
    const int r = lane;
    float F = 0.f;
#pragma unroll
    for (int i = 0; i < NW; ++i) F += scal[i][0];
    const float e1 = rowacc[0][0][r] + rowacc[1][0][r];
    const float e2 = rowacc[0][1][r] + rowacc[1][1][r];
    const float bl = rowacc[0][2][r] + rowacc[1][2][r];
    const float p1 = rowacc[0][3][r] + rowacc[1][3][r];
    const float p2 = rowacc[0][4][r] + rowacc[1][4][r];
    const float p3 = rowacc[0][5][r] + rowacc[1][5][r];
    const float col = colpart[0][r] + colpart[1][r] + colpart[2][r] + colpart[3][r];
    const float egm = __expf(r > 0 ? Gs[r - 1] : 0.f);
    const float cr = __expf(Glast - Gs[r]) * p2;
    const float rowg = e1 + __expf(Gs[r]) * p1 - cr;
    const float rowgm = e2 - Bts[r] * egm * p3;
    const float rowbt = bl - egm * p3;  // through beta~
    const float gcs = wave_sum(cr);
    const float rowgm_next = shift_down1(rowgm);
    float dG = rowg - col + (r + 1 < CH ? rowgm_next : 0.f);
    if (r == CH - 1) dG += gcs + __expf(Glast) * F;
    float x = __shfl(dG, 63 - lane);
    x = wave_prefix_sum(x);
    const float dgr = __shfl(x, 63 - lane);
    if (r < len) {
      at(dg + tok, 4u * (r * H)) = dgr;
      if (dbeta_tilde) {
        at(dbeta + tok, 4u * (r * H)) = rowB[r];
        at(dbeta_tilde + tok, 4u * (r * H)) = rowbt;
      } else {
        at(dbeta + tok, 4u * (r * H)) = rowB[r] + rowbt;
      }
    }
  }

  // dQ~ (in T1) and dK (in T2)
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int r = 16 * rt + 4 * g4 + e;
    const float gr = __expf(rv.g[e]), dec = __expf(Glast - rv.g[e]);
    const float sr = rv.bt[e] * __expf(r > 0 ? rv.gm[e] : 0.f);
#pragma unroll
    for (int j = 0; j < NTW; ++j) {
      T1[j][e] *= gr;
      T2[j][e] = dec * T2[j][e] - sr * T3[j][e];
    }
  }
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    // A operands of this wave's rows x = 16 rt + r16: G and P rows via
    // transposing reads of GT, PT; G^T and U rows directly
    const int ar = (16 * rt + r16) * LDC + 32 * ks + 8 * g4;
    const bf16x8 agh = ld_tr8(GTh, LDC, 32 * ks + 8 * g4, 16 * rt);
    const bf16x8 agl = ld_tr8(GTl, LDC, 32 * ks + 8 * g4, 16 * rt);
    const bf16x8 aph = ld_tr8(PTh, LDC, 32 * ks + 8 * g4, 16 * rt);
    const bf16x8 apl = ld_tr8(PTl, LDC, 32 * ks + 8 * g4, 16 * rt);
    const bf16x8 ath = ld8(GTh + ar), atl = ld8(GTl + ar);
    const bf16x8 auh = ld8(Ubh + ar), aul = ld8(Ubl + ar);
#pragma unroll
    for (int j = 0; j < NTW; ++j) {
      // B operands K^T, Q^T of this wave's dk columns, B(k = t, n = c) = K[t][c],
      // read transposed from the row-major LDS tiles
      const bf16x8 ktb = ld_tr8(Ks, LDK, 32 * ks + 8 * g4, 16 * (ch * NTW + j));
      const bf16x8 qtb = ld_tr8(Qs, LDK, 32 * ks + 8 * g4, 16 * (ch * NTW + j));
      T1[j] = mfma16(agh, ktb, T1[j]);
      T1[j] = mfma16(agl, ktb, T1[j]);
      T2[j] = mfma16(ath, qtb, T2[j]);
      T2[j] = mfma16(atl, qtb, T2[j]);
      T2[j] = mfma16(aph, ktb, T2[j]);
      T2[j] = mfma16(apl, ktb, T2[j]);
      T2[j] = mfma16(auh, ktb, T2[j]);
      T2[j] = mfma16(aul, ktb, T2[j]);
    }
  }
  float ddpart = 0.f;
  // this chunk's rows (row r at r H DK), bounded at row len
  const __amdgpu_buffer_rsrc_t rq = clip_rsrc(dq + tok * DK, (unsigned)len * (unsigned)(H * DK * 4));
  const __amdgpu_buffer_rsrc_t rk = clip_rsrc(dk + tok * DK, (unsigned)len * (unsigned)(H * DK * 4));
#pragma unroll
  for (int j = 0; j < NTW; ++j) {
    floatx4 dkv;
    const bf16x4_t k4 = ld_tr4(Ks, LDK, 16 * rt + 4 * g4, 16 * (ch * NTW + j));
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float dqt = T1[j][e];
      ddpart += (float)k4[e] * dqt;
      dkv[e] = T2[j][e] - dh * dqt;
    }
    // straight from the accumulators (16 lanes write 64 contiguous bytes of a
    // row): transposing to 16-byte pieces first costs more VALU than it saves
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = 16 * rt + 4 * g4 + e;
      const unsigned off = 4u * ((unsigned)r * (H * DK) + 16 * (ch * NTW + j) + r16);
      store_clip(T1[j][e], rq, off);  // rows r >= len dropped
      store_clip(dkv[e], rk, off);
    }
  }
  {
    // The next item's gates and beta, after this item's last loads and stores:
    // a wait for them (in-order counters) is then a wait for everything, so
    // they must not be needed earlier.  Unconditional, from a clamped item and
    // row (this item has tokens, so every such address is valid): behind a
    // branch, the merge would copy them and wait right there.
    const int nxc = min(item + (int)gridDim.x, nitems - 1);
    const ChunkInfo ci2 = chunk_at(cmap, nxc % ncmax, Tfix);
    const int h2 = nxc / ncmax;
    const long chh2 = (long)(nxc % ncmax) * H + h2, tok2 = (long)ci2.tok0 * H + h2;
    g_nx = Gw[chh2 * CH + (tid & (CH - 1))];
    const long brow2 = tok2 + (long)min(tid & (CH - 1), max(ci2.len, 1) - 1) * H;
    b_nx = beta[brow2];
    bt_nx = beta_tilde[brow2];
  }
  ddpart = wave_sum(ddpart);
  if (lane == 0) scal[w][1] = ddpart;
  __syncthreads();
  if (w == 0 && lane == 0) {
    float dds = 0.f;
#pragma unroll
    for (int i = 0; i < NW; ++i) dds += scal[i][1];
    ddp[chh] = -dds;
  }
  __syncthreads();  // the next item rewrites Gs, Bs
  }
  // no copy into R0 may still be in flight when the workgroup ends
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// ---------------------------------------------------------------------------
// k_intra_bwd_wide: the intra-chunk gradients at head dim 256 (dk = 256).  The
// work of k_intra_bwd_bf in dk / 128 passes over 128-wide slices of dk, so that
// the LDS tiles and the T1, T2, T3 accumulators keep their dk = 128 size.  Every
// quantity that spans dk enters the row and column sums linearly (the K K^T and
// Q K^T terms of E1, E2, BL, the row dots p1, p2, p3, <X, Y>, <k, dQ~>), so each
// pass adds its part and the sums are combined at the end; dA, dL, <v, dR> and
// dv do not involve dk and are formed in the first pass.  One workgroup per
// chunk-head (no persistent loop, no next-item copy).
// ---------------------------------------------------------------------------
template <int DK, int DV>
__global__ __launch_bounds__(IB_THR, 1) void k_intra_bwd_wide(
    const bf16_t* __restrict__ q, const bf16_t* __restrict__ k, const bf16_t* __restrict__ v,
    const bf16_t* __restrict__ dO, const bf16_t* __restrict__ beta,
    const bf16_t* __restrict__ beta_tilde, const float* __restrict__ d,
    const ChunkInfo* __restrict__ cmap, int Tfix, int H, const float* __restrict__ Gw,
    const int16_t* __restrict__ Xq, const float* __restrict__ Xs, const int16_t* __restrict__ Dq,
    const float* __restrict__ Ds, const int16_t* __restrict__ Yq, const float* __restrict__ Ys,
    const int16_t* __restrict__ dRq, const float* __restrict__ dRs, float* __restrict__ dq,
    float* __restrict__ dk, float* __restrict__ dv, float* __restrict__ dbeta,
    float* __restrict__ dbeta_tilde, float* __restrict__ dg, float* __restrict__ ddp) {
  constexpr int DKP = 128, KP = DK / DKP;
  static_assert(DK % DKP == 0, "dk slices");
  using SM = IntraBwdBfSmem<DKP>;
  constexpr int VB = SM::VB, LDB = SM::LDB, LDK = SM::LDK, LDC = SM::LDC;
  constexpr int NTW = DKP / 32;
  constexpr int NW = IB_THR / 64;
  constexpr int NVB = DV / VB;
  constexpr int XP = DKP * (VB / 4) / IB_THR;
  constexpr int NB = DV / 32;
  static_assert(VB == 32 && NVB % 2 == 0 && CH * 8 == IB_THR, "blocks and pieces");
  __shared__ __align__(16) char smem[SM::BYTES];
  __shared__ __align__(16) float Gs[CH], Bs[CH], Bts[CH], rowB[CH];
  __shared__ float colpart[KP][4][CH];
  __shared__ float rowacc[KP][2][6][CH];
  __shared__ float scal[KP][NW][2];

  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, r16 = lane & 15, g4 = lane >> 4;
  const int rt = w & 3, ch = w >> 2;
  const int h = blockIdx.y;
  const long chh = (long)blockIdx.x * H + h;
  const ChunkInfo ci = chunk_at(cmap, blockIdx.x, Tfix);
  if (ci.len <= 0) {
    if (tid == 0) ddp[chh] = 0.f;
    return;
  }
  const long tok = (long)ci.tok0 * H + h;
  const int len = ci.len;
  const float dh = d[h];
  if (tid < CH) {
    const long row = tok + (long)min(tid, len - 1) * H;
    Gs[tid] = Gw[chh * CH + tid];
    Bs[tid] = tid < len ? bf2f(beta[row]) : 0.f;
    Bts[tid] = tid < len ? bf2f(beta_tilde[row]) : 0.f;
  }

  bf16_t* dOb = reinterpret_cast<bf16_t*>(smem);
  bf16_t* dRh = dOb + CH * LDB;
  bf16_t* dRl = dRh + CH * LDB;
  bf16_t* Dh = dRl + CH * LDB;
  bf16_t* Dl = Dh + CH * LDB;
  bf16_t* Xh = Dl + CH * LDB;
  bf16_t* Xl = Xh + DKP * LDB;
  bf16_t* Yh = Xl + DKP * LDB;
  bf16_t* Yl = Yh + DKP * LDB;
  bf16_t* Vb = Yl + DKP * LDB;
  const int pr = tid >> 3, pc = (tid & 7) * 8, pb = (tid & 7) >> 2;
  const int pf_r = tid >> 3, pf_c = (tid & 7) * 4;
  uint4 r_do, r_v;
  uint2 r_dr, r_d, r_x[XP], r_y[XP];
  float s_dr, s_d, s_x[XP], s_y[XP];
  const bf16_t* dO_i = dO + tok * DV;
  const bf16_t* v_i = v + tok * DV;
  const int16_t* dRq_i = dRq + chh * NB * CH * VB;
  const int16_t* Dq_i = Dq + chh * NB * CH * VB;
  const float* dRs_i = dRs + chh * NB * CH;
  const float* Ds_i = Ds + chh * NB * CH;
  const int16_t* Xq_i = Xq + chh * NB * DK * VB;  // [block][dk rows][32]
  const int16_t* Yq_i = Yq + chh * NB * DK * VB;
  const float* Xs_i = Xs + chh * NB * DK;
  const float* Ys_i = Ys + chh * NB * DK;
  // this chunk's dv rows (row r at r H DV), bounded at row len
  const __amdgpu_buffer_rsrc_t rdv = clip_rsrc(dv + tok * DV, (unsigned)len * (unsigned)(H * DV * 4));
  // this chunk's rows (row r at r H DK), bounded at row len
  const __amdgpu_buffer_rsrc_t rq = clip_rsrc(dq + tok * DK, (unsigned)len * (unsigned)(H * DK * 4));
  const __amdgpu_buffer_rsrc_t rk = clip_rsrc(dk + tok * DK, (unsigned)len * (unsigned)(H * DK * 4));
  floatx4 dA[2], dL[2];
  dA[0] = dA[1] = dL[0] = dL[1] = zero4();
  float bv = 0.f;
  float4 fdr;

  // block vb of pass kh (its dk columns kh DKP .. + 127) into the registers
  auto issue = [&](int kh, int vb) {
    const int c0 = kh * DKP;
      if (vb % 2 == 0) {
        const unsigned rb = 2u * ((unsigned)min(pr, len - 1) * (H * DV) + vb * VB + pc);
        r_do = at(reinterpret_cast<const uint4*>(dO_i), rb);
        r_v = at(reinterpret_cast<const uint4*>(v_i), rb);
      }
      const unsigned rr = vb * CH + pf_r;
      r_dr = at(reinterpret_cast<const uint2*>(dRq_i), 2u * (rr * VB + pf_c));
      r_d = at(reinterpret_cast<const uint2*>(Dq_i), 2u * (rr * VB + pf_c));
      s_dr = at(dRs_i, 4u * rr);
      s_d = at(Ds_i, 4u * rr);
#pragma unroll
      for (int p = 0; p < XP; ++p) {
        const int pc2 = tid + p * IB_THR, xr = pc2 >> 3, xc = (pc2 & 7) * 4;
        const unsigned xrow = vb * DK + c0 + xr;
        r_x[p] = at(reinterpret_cast<const uint2*>(Xq_i), 2u * (xrow * VB + xc));
        r_y[p] = at(reinterpret_cast<const uint2*>(Yq_i), 2u * (xrow * VB + xc));
        s_x[p] = at(Xs_i, 4u * xrow);
        s_y[p] = at(Ys_i, 4u * xrow);
      }
  };
  issue(0, 0);
  for (int kh = 0; kh < KP; ++kh) {
    const int c0 = kh * DKP;  // this pass's dk columns c0 .. c0 + 127
    float Fpart = 0.f;
    auto put = [&](int vb) {
      const int j = vb * VB;
      if (pb == (vb & 1)) {
        *reinterpret_cast<uint4*>(dOb + pr * LDB + (pc & 31)) = r_do;
        *reinterpret_cast<uint4*>(Vb + pr * LDB + (pc & 31)) = r_v;
      }
      bf16x4 hh, ll;
      fdr = q_unpack4(r_dr, s_dr);
      split4v(fdr, hh, ll);
      *reinterpret_cast<bf16x4*>(dRh + pf_r * LDB + pf_c) = hh;
      *reinterpret_cast<bf16x4*>(dRl + pf_r * LDB + pf_c) = ll;
      split4v(q_unpack4(r_d, s_d), hh, ll);
      *reinterpret_cast<bf16x4*>(Dh + pf_r * LDB + pf_c) = hh;
      *reinterpret_cast<bf16x4*>(Dl + pf_r * LDB + pf_c) = ll;
#pragma unroll
      for (int p = 0; p < XP; ++p) {
        const int pc2 = tid + p * IB_THR, xr = pc2 >> 3, xc = (pc2 & 7) * 4;
        const float4 fx = q_unpack4(r_x[p], s_x[p]), fy = q_unpack4(r_y[p], s_y[p]);
        split4v(fx, hh, ll);
        *reinterpret_cast<bf16x4*>(Xh + xr * LDB + xc) = hh;
        *reinterpret_cast<bf16x4*>(Xl + xr * LDB + xc) = ll;
        split4v(fy, hh, ll);
        *reinterpret_cast<bf16x4*>(Yh + xr * LDB + xc) = hh;
        *reinterpret_cast<bf16x4*>(Yl + xr * LDB + xc) = ll;
        Fpart += fx.x * fy.x + fx.y * fy.y + fx.z * fy.z + fx.w * fy.w;
      }
      if (kh == 0) {  // dv = Diag(beta) dR, once
        const float b = Bs[pf_r];
        store_clip4(floatx4{b * fdr.x, b * fdr.y, b * fdr.z, b * fdr.w}, rdv,
                    4u * ((unsigned)pf_r * (H * DV) + j + pf_c));  // rows >= len dropped
      }
    };

    floatx4 T1[NTW], T2[NTW], T3[NTW];
#pragma unroll
    for (int j = 0; j < NTW; ++j) T1[j] = T2[j] = T3[j] = zero4();
    TileRegs<bf16_t, CH, DKP, IB_THR> kr, qr;
    // one block per iteration: unrolled, the blocks of dv = 256 keep too many
    // loaded pieces live and spill
#pragma unroll 1
    for (int vb = 0; vb < NVB; ++vb) {
      __syncthreads();
      put(vb);
      __syncthreads();
      if (vb + 1 < NVB) {
        issue(kh, vb + 1);
      } else {
        kr.load_clip(k + tok * DK + c0, (long)H * DK, len);
        qr.load_clip(q + tok * DK + c0, (long)H * DK, len);
      }
      if (kh == 0) {
        const bf16x4 vv = *reinterpret_cast<const bf16x4*>(Vb + pf_r * LDB + pf_c);
        bv += (float)vv[0] * fdr.x + (float)vv[1] * fdr.y + (float)vv[2] * fdr.z + (float)vv[3] * fdr.w;
      }
      const int arow = (16 * rt + r16) * LDB + 8 * g4;
      bf16x8 a_do = ld8(dOb + arow);
      if (16 * rt + r16 >= len) a_do = bf16x8{};
      const bf16x8 a_drh = ld8(dRh + arow), a_drl = ld8(dRl + arow);
      const bf16x8 a_dh = ld8(Dh + arow), a_dl = ld8(Dl + arow);
#pragma unroll
      for (int j = 0; j < NTW; ++j) {
        const int brow = (16 * (ch * NTW + j) + r16) * LDB + 8 * g4;
        const bf16x8 xh = ld8(Xh + brow), xl = ld8(Xl + brow);
        const bf16x8 yh = ld8(Yh + brow), yl = ld8(Yl + brow);
        T1[j] = mfma16(a_do, xh, T1[j]);
        T1[j] = mfma16(a_do, xl, T1[j]);
        T3[j] = mfma16(a_drh, xh, T3[j]);
        T3[j] = mfma16(a_drh, xl, T3[j]);
        T3[j] = mfma16(a_drl, xh, T3[j]);
        T2[j] = mfma16(a_dh, yh, T2[j]);
        T2[j] = mfma16(a_dh, yl, T2[j]);
        T2[j] = mfma16(a_dl, yh, T2[j]);
      }
      if (kh == 0) {
#pragma unroll
        for (int j2 = 0; j2 < 2; ++j2) {
          const int brow = (16 * (2 * ch + j2) + r16) * LDB + 8 * g4;
          const bf16x8 bh = ld8(Dh + brow), bl = ld8(Dl + brow);
          dA[j2] = mfma16(a_do, bh, dA[j2]);
          dA[j2] = mfma16(a_do, bl, dA[j2]);
          dL[j2] = mfma16(a_drh, bh, dL[j2]);
          dL[j2] = mfma16(a_drh, bl, dL[j2]);
          dL[j2] = mfma16(a_drl, bh, dL[j2]);
        }
      }
    }
    if (kh == 0) {
      bv = sum8(bv);
      if ((tid & 7) == 0) rowB[pf_r] = bv;
    }
    Fpart = wave_sum(Fpart);
    if (lane == 0) scal[kh][w][0] = Fpart;
    __syncthreads();

    // ---- phase 2 of the pass ----
    bf16_t* Ks = reinterpret_cast<bf16_t*>(smem);
    bf16_t* Qs = Ks + CH * LDK;
    bf16_t* GTh = Qs + CH * LDK;
    bf16_t* GTl = GTh + CH * LDC;
    bf16_t* PTh = GTl + CH * LDC;
    bf16_t* PTl = PTh + CH * LDC;
    bf16_t* Ubh = PTl + CH * LDC;
    bf16_t* Ubl = Ubh + CH * LDC;
    kr.store(Ks, LDK);
    qr.store(Qs, LDK);
    __syncthreads();
    // the next pass's first block loads during this phase 2 (it reads nothing
    // else from memory)
    if (kh + 1 < KP) issue(kh + 1, 0);
    const float Glast = Gs[CH - 1];
    const RowVals rv = row_vals(Gs, Bts, 16 * rt + 4 * g4);
    {
      floatx4 akk[2], aqk[2];
      akk[0] = akk[1] = aqk[0] = aqk[1] = zero4();
#pragma unroll
      for (int ks = 0; ks < DKP / 32; ++ks) {
        const int ar = (16 * rt + r16) * LDK + 32 * ks + 8 * g4;
        const bf16x8 a_k = ld8(Ks + ar), a_q = ld8(Qs + ar);
#pragma unroll
        for (int j2 = 0; j2 < 2; ++j2) {
          const bf16x8 b = ld8(Ks + (16 * (2 * ch + j2) + r16) * LDK + 32 * ks + 8 * g4);
          akk[j2] = mfma16(a_k, b, akk[j2]);
          aqk[j2] = mfma16(a_q, b, aqk[j2]);
        }
      }
      float rE1[4] = {0.f, 0.f, 0.f, 0.f}, rE2[4] = {0.f, 0.f, 0.f, 0.f}, rBL[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j2 = 0; j2 < 2; ++j2) {
        const int c = 16 * (2 * ch + j2) + r16;
        const float Gc = Gs[c];
        float cE = 0.f, dagv[4], pv[4], uv[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          // akk: this pass's part of k_r . k_c
          const GateTerms t = gate_terms(16 * rt + 4 * g4 + e, c, rv, e, Gc, akk[j2][e], aqk[j2][e],
                                         dA[j2][e], dL[j2][e], dh, rBL[e]);
          dagv[e] = t.dag;
          pv[e] = t.dakk;
          uv[e] = t.dakk - dh * t.dag;
          rE1[e] += t.e1;
          rE2[e] += t.e2;
          cE += t.e1 + t.e2;
        }
        const int toff = c * LDC + 16 * rt + 4 * g4;
        put_t4(GTh, GTl, toff, dagv);
        put_t4(PTh, PTl, toff, pv);
        put_t4(Ubh, Ubl, toff, uv);
        cE = sum_groups(cE);
        if (g4 == 0) colpart[kh][rt][c] = cE;
      }
      float p1[4] = {0.f, 0.f, 0.f, 0.f}, p2[4] = {0.f, 0.f, 0.f, 0.f}, p3[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < NTW; ++j) {
        const bf16x4_t k4 = ld_tr4(Ks, LDK, 16 * rt + 4 * g4, 16 * (ch * NTW + j));
        const bf16x4_t q4 = ld_tr4(Qs, LDK, 16 * rt + 4 * g4, 16 * (ch * NTW + j));
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float kv = (float)k4[e];
          const float qv = (float)q4[e] - dh * kv;
          p1[e] += T1[j][e] * qv;
          p2[e] += T2[j][e] * kv;
          p3[e] += T3[j][e] * kv;
        }
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float s0 = sum16(rE1[e]), s1 = sum16(rE2[e]), s2 = sum16(rBL[e]);
        const float s3 = sum16(p1[e]), s4 = sum16(p2[e]), s5 = sum16(p3[e]);
        if (r16 == 0) {
          const int r = 16 * rt + 4 * g4 + e;
          rowacc[kh][ch][0][r] = s0;
          rowacc[kh][ch][1][r] = s1;
          rowacc[kh][ch][2][r] = s2;
          rowacc[kh][ch][3][r] = s3;
          rowacc[kh][ch][4][r] = s4;
          rowacc[kh][ch][5][r] = s5;
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = 16 * rt + 4 * g4 + e;
      const float gr = __expf(rv.g[e]), dec = __expf(Glast - rv.g[e]);
      const float sr = rv.bt[e] * __expf(r > 0 ? rv.gm[e] : 0.f);
#pragma unroll
      for (int j = 0; j < NTW; ++j) {
        T1[j][e] *= gr;
        T2[j][e] = dec * T2[j][e] - sr * T3[j][e];
      }
    }
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int ar = (16 * rt + r16) * LDC + 32 * ks + 8 * g4;
      const bf16x8 agh = ld_tr8(GTh, LDC, 32 * ks + 8 * g4, 16 * rt);
      const bf16x8 agl = ld_tr8(GTl, LDC, 32 * ks + 8 * g4, 16 * rt);
      const bf16x8 aph = ld_tr8(PTh, LDC, 32 * ks + 8 * g4, 16 * rt);
      const bf16x8 apl = ld_tr8(PTl, LDC, 32 * ks + 8 * g4, 16 * rt);
      const bf16x8 ath = ld8(GTh + ar), atl = ld8(GTl + ar);
      const bf16x8 auh = ld8(Ubh + ar), aul = ld8(Ubl + ar);
#pragma unroll
      for (int j = 0; j < NTW; ++j) {
        const bf16x8 ktb = ld_tr8(Ks, LDK, 32 * ks + 8 * g4, 16 * (ch * NTW + j));
        const bf16x8 qtb = ld_tr8(Qs, LDK, 32 * ks + 8 * g4, 16 * (ch * NTW + j));
        T1[j] = mfma16(agh, ktb, T1[j]);
        T1[j] = mfma16(agl, ktb, T1[j]);
        T2[j] = mfma16(ath, qtb, T2[j]);
        T2[j] = mfma16(atl, qtb, T2[j]);
        T2[j] = mfma16(aph, ktb, T2[j]);
        T2[j] = mfma16(apl, ktb, T2[j]);
        T2[j] = mfma16(auh, ktb, T2[j]);
        T2[j] = mfma16(aul, ktb, T2[j]);
      }
    }
    float ddpart = 0.f;
#pragma unroll
    for (int j = 0; j < NTW; ++j) {
      floatx4 dkv;
      const bf16x4_t k4 = ld_tr4(Ks, LDK, 16 * rt + 4 * g4, 16 * (ch * NTW + j));
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float dqt = T1[j][e];
        ddpart += (float)k4[e] * dqt;
        dkv[e] = T2[j][e] - dh * dqt;
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 16 * rt + 4 * g4 + e;
        const unsigned off = 4u * ((unsigned)r * (H * DK) + c0 + 16 * (ch * NTW + j) + r16);
        store_clip(T1[j][e], rq, off);  // rows r >= len dropped
        store_clip(dkv[e], rk, off);
      }
    }
    ddpart = wave_sum(ddpart);
    if (lane == 0) scal[kh][w][1] = ddpart;
    __syncthreads();  // the next pass rewrites the LDS tiles
  }

  if (w == 0) {
    const int r = lane;
    float F = 0.f, dds = 0.f, e1 = 0.f, e2 = 0.f, bl = 0.f, p1 = 0.f, p2 = 0.f, p3 = 0.f, col = 0.f;
#pragma unroll
    for (int kh = 0; kh < KP; ++kh) {
#pragma unroll
      for (int i = 0; i < NW; ++i) {
        F += scal[kh][i][0];
        dds += scal[kh][i][1];
      }
#pragma unroll
      for (int c2 = 0; c2 < 2; ++c2) {
        e1 += rowacc[kh][c2][0][r];
        e2 += rowacc[kh][c2][1][r];
        bl += rowacc[kh][c2][2][r];
        p1 += rowacc[kh][c2][3][r];
        p2 += rowacc[kh][c2][4][r];
        p3 += rowacc[kh][c2][5][r];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) col += colpart[kh][i][r];
    }
    const float Glast = Gs[CH - 1];
    const float egm = __expf(r > 0 ? Gs[r - 1] : 0.f);
    const float cr = __expf(Glast - Gs[r]) * p2;
    const float rowg = e1 + __expf(Gs[r]) * p1 - cr;
    const float rowgm = e2 - Bts[r] * egm * p3;
    const float rowbt = bl - egm * p3;
    const float gcs = wave_sum(cr);
    const float rowgm_next = shift_down1(rowgm);
    float dG = rowg - col + (r + 1 < CH ? rowgm_next : 0.f);
    if (r == CH - 1) dG += gcs + __expf(Glast) * F;
    float x = __shfl(dG, 63 - lane);
    x = wave_prefix_sum(x);
    const float dgr = __shfl(x, 63 - lane);
    if (r < len) {
      at(dg + tok, 4u * (r * H)) = dgr;
      if (dbeta_tilde) {
        at(dbeta + tok, 4u * (r * H)) = rowB[r];
        at(dbeta_tilde + tok, 4u * (r * H)) = rowbt;
      } else {
        at(dbeta + tok, 4u * (r * H)) = rowB[r] + rowbt;
      }
    }
    if (lane == 0) ddp[chh] = -dds;
  }
}

// ---------------------------------------------------------------------------
// host launchers
// ---------------------------------------------------------------------------
// Compute units of the current device (0 when the query fails).
static int device_cus() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  return cus > 0 ? cus : 0;
}

// Workgroups of the persistent k_intra_bwd_bf: one per CU (all items when the
// CU count is unavailable).
static unsigned intra_bwd_grid(long items) {
  const int cus = device_cus();
  return (unsigned)(cus > 0 && cus < items ? cus : items);
}

// Work that can run beside the caller's stream: a second stream per device
// (default priority, non-blocking, created on first use and kept until the
// process ends) with a fork and a join event.  side(st) enqueues, in order, a
// fork (the side stream waits for everything already on st), the side work,
// the main work on st and a join (st waits for the side work), under a lock,
// so that calls from several host threads cannot interleave their event
// records.  Without a side stream (creation failed, or the first use falls
// in a graph capture of st) both run on st in turn.  Under graph capture of
// st an existing side stream joins the capture and rejoins st.
struct SideStream {
  hipStream_t s = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
  bool failed = false;
};
constexpr int kMaxSideDevices = 64;
static std::mutex g_side_mu;
static SideStream g_side[kMaxSideDevices];

template <typename Main, typename Side>
static void side(hipStream_t st, Main&& main_work, Side&& side_work) {
  int dev = 0;
  SideStream* ss = nullptr;
  // an error left by the side stream's own calls is cleared (the work then
  // runs in turn), unless one was already pending from the caller's launches
  const bool clean = hipPeekAtLastError() == hipSuccess;
  std::unique_lock<std::mutex> lock(g_side_mu);
  if (hipGetDevice(&dev) == hipSuccess && dev >= 0 && dev < kMaxSideDevices) {
    SideStream& c = g_side[dev];
    // creating a stream or an event is not allowed while st is being captured:
    // then the work runs in turn (an existing side stream forks and joins as
    // usual: event records and waits are captured)
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    bool capturing = false;
    if (!c.s && !c.failed) {
      if (hipStreamIsCapturing(st, &cs) == hipSuccess)
        capturing = cs != hipStreamCaptureStatusNone;
      else if (clean)
        (void)hipGetLastError();  // no capture to be found on this stream
    }
    if (!c.s && !c.failed && !capturing) {
      if (hipStreamCreateWithFlags(&c.s, hipStreamNonBlocking) != hipSuccess ||
          hipEventCreateWithFlags(&c.fork, hipEventDisableTiming) != hipSuccess ||
          hipEventCreateWithFlags(&c.join, hipEventDisableTiming) != hipSuccess) {
        c.failed = true;  // run in turn from now on
        c.s = nullptr;
      }
    }
    if (c.s) ss = &c;
  }
  if (!ss || hipEventRecord(ss->fork, st) != hipSuccess ||
      hipStreamWaitEvent(ss->s, ss->fork, 0) != hipSuccess) {
    if (clean) (void)hipGetLastError();
    main_work(st);
    side_work(st);
    return;
  }
  side_work(ss->s);
  main_work(st);
  if (hipEventRecord(ss->join, ss->s) != hipSuccess || hipStreamWaitEvent(st, ss->join, 0) != hipSuccess)
    (void)hipStreamSynchronize(ss->s);  // keep the order on the host if the join cannot be enqueued
}

// 1-D grid of the bf16 scans: whole groups of 8 chains (see scan_item).
static unsigned scan_blocks(int N, int H, int nsl) {
  return (unsigned)((((long)N * H + 7) / 8) * 8 * nsl);
}

// Sequence and chunk tables: the per-sequence scan (one workgroup), then one
// thread per chunk slot.
static void launch_chunk_map(const LaunchArgs& a, hipStream_t st) {
  k_seq_map<<<1, NTHR, 0, st>>>(a.cu_seqlens, a.N, a.Tseq, a.Ttot, a.ncmax, a.smap, a.sorder);
  if (a.ncmax > 0) {
    const int blocks = (a.ncmax + NTHR - 1) / NTHR;
    k_chunk_fill<<<blocks < 1024 ? blocks : 1024, NTHR, 0, st>>>(a.smap, a.N, a.ncmax, a.cmap);
  }
}

template <typename Tin, int DK, int DV>
static hipError_t run_fwd(const LaunchArgs& a) {
  hipStream_t st = a.stream;
  const Tin* q = static_cast<const Tin*>(a.q);
  const Tin* k = static_cast<const Tin*>(a.k);
  const Tin* v = static_cast<const Tin*>(a.v);
  const Tin* beta = static_cast<const Tin*>(a.beta);
  const Tin* bt = static_cast<const Tin*>(a.beta_tilde);
  a.stage("chunk_map");
  launch_chunk_map(a, st);
  a.stage("prep");
  if (a.ncmax > 0)
    k_prep<Tin, DK><<<dim3(a.ncmax, a.H), NTHR, 0, st>>>(q, k, a.g, bt, a.d, a.cmap, a.H, a.Mw,
                                                         a.Aw, a.Gw);
  a.stage("scan_fwd");
  if (a.saved)
    k_scan_fwd<Tin, DK, DV, true, true><<<dim3(a.N, a.H, DV / 32), NTHR, 0, st>>>(
        q, k, v, beta, bt, a.d, a.h0, a.cmap, a.smap, a.H, a.Mw, a.Aw, a.Gw, a.o, a.ht, a.Xw, a.Dw);
  else
    k_scan_fwd<Tin, DK, DV, true, false><<<dim3(a.N, a.H, DV / 32), NTHR, 0, st>>>(
        q, k, v, beta, bt, a.d, a.h0, a.cmap, a.smap, a.H, a.Mw, a.Aw, a.Gw, a.o, a.ht, nullptr,
        nullptr);
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
  const Tin* bt = static_cast<const Tin*>(a.beta_tilde);
  const Tin* dO = static_cast<const Tin*>(a.dO);
  if (a.N == 0) {
    // no sequences: dd (one value per head) is zero
    k_reduce_dd<<<a.H, RDD_THR, 0, st>>>(a.ddp, 0, a.H, a.dd);
    return hipGetLastError();
  }
  if (!a.saved) {
    a.stage("chunk_map");
    launch_chunk_map(a, st);
    a.stage("prep");
    if (a.ncmax > 0)
      k_prep<Tin, DK><<<dim3(a.ncmax, a.H), NTHR, 0, st>>>(q, k, a.g, bt, a.d, a.cmap, a.H,
                                                           a.Mw, a.Aw, a.Gw);
    a.stage("scan_fwd_store");
    k_scan_fwd<Tin, DK, DV, false, true><<<dim3(a.N, a.H, DV / 32), NTHR, 0, st>>>(
        q, k, v, beta, bt, a.d, a.h0, a.cmap, a.smap, a.H, a.Mw, a.Aw, a.Gw, nullptr, nullptr, a.Xw,
        a.Dw);
  }
  a.stage("scan_bwd");
  k_scan_bwd<Tin, DK, DV><<<dim3(a.N, a.H, DV / 32), NTHR, 0, st>>>(
      q, k, dO, bt, a.d, a.dht, a.cmap, a.smap, a.H, a.Mw, a.Aw, a.Gw, a.dh0, a.Yw, a.dRw);
  a.stage("intra_bwd");
  if (a.ncmax > 0)
    k_intra_bwd<Tin, DK, DV><<<dim3(a.ncmax, a.H), NTHR, 0, st>>>(
        q, k, v, dO, beta, bt, a.d, a.cmap, a.H, a.Gw, a.Xw, a.Dw, a.Yw, a.dRw, a.dq, a.dk_, a.dv_,
        a.dbeta, a.dbeta_tilde, a.dg, a.ddp);
  a.stage("reduce_dd");
  k_reduce_dd<<<a.H, RDD_THR, 0, st>>>(a.ddp, a.ncmax, a.H, a.dd);
  a.stage(nullptr);
  return hipGetLastError();
}

// The segmented scans' state passes and boundary states (see run_fwd_bf):
// each segment's final state from a zero start (not of a row's last segment),
// its transition product (of every segment when a backward follows, which
// needs those of all but the first; else not of the last) and the true state
// entering every segment.
// vsm, Tv: the virtual rows (packed sequences: the table of k_seg_map, Tv < 0;
// fixed-length rows: vsm NULL, Tv = Tseq / P tokens each).
template <int DK, int DV>
static void seg_forward_states(const LaunchArgs& a, const bf16_t* q, const bf16_t* k,
                               const bf16_t* v, const bf16_t* beta, const bf16_t* bt,
                               bool phi_all, const SeqInfo* vsm, int Tp) {
  hipStream_t st = a.stream;
  const int P = a.segP, Nst = a.N * (P - 1);
  const int Nphi = phi_all ? a.N * P : Nst, gphi = phi_all ? 0 : P;
  a.stage("scan_seg_state");
  k_scan_fwd_bf<DK, DV, SCAN_BV, false, false><<<scan_blocks(Nst, a.H, DV / SCAN_BV), NTHR, 0, st>>>(
      q, k, v, beta, bt, a.d, nullptr, vsm, nullptr, Nst, Tp, a.H, a.Mq, a.Ms, a.Aq, a.As, a.Gw,
      nullptr, a.segF, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, P);
  a.stage("scan_seg_phi");
  k_scan_fwd_bf<DK, DK, SCAN_BV, false, false, true><<<scan_blocks(Nphi, a.H, DK / SCAN_BV), NTHR, 0, st>>>(
      q, k, v, beta, bt, a.d, nullptr, vsm, nullptr, Nphi, Tp, a.H, a.Mq, a.Ms, a.Aq, a.As, a.Gw,
      nullptr, a.segPhi, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, gphi);
  a.stage("seg_combine");
  k_seg_combine<DK, DV><<<a.N * a.H * (DV / SEG_SL), NTHR, 0, st>>>(a.segPhi, a.segF, a.h0, P, a.H,
                                                                a.segX0);
}

// Row r's state from virtual row r P + p (p = 0: the first segment's, P - 1:
// the last's) into dst [N, H, dk, dv].
template <int DK, int DV>
static hipError_t seg_copy_rows(const LaunchArgs& a, float* dst, const float* src, int p) {
  const size_t st_bytes = (size_t)a.H * DK * DV * sizeof(float);
  return hipMemcpy2DAsync(dst, st_bytes, src + (size_t)p * a.H * DK * DV, a.segP * st_bytes,
                          st_bytes, a.N, hipMemcpyDeviceToDevice, a.stream);
}

template <int DK, int DV>
static hipError_t run_fwd_bf(const LaunchArgs& a) {
  hipStream_t st = a.stream;
  const bf16_t* q = static_cast<const bf16_t*>(a.q);
  const bf16_t* k = static_cast<const bf16_t*>(a.k);
  const bf16_t* v = static_cast<const bf16_t*>(a.v);
  const bf16_t* beta = static_cast<const bf16_t*>(a.beta);
  const bf16_t* bt = static_cast<const bf16_t*>(a.beta_tilde);
  // fixed-length rows need no tables (closed form in the kernels)
  const int Tfix = a.cu_seqlens ? -1 : a.Tseq;
  const int* sord = Tfix < 0 ? a.sorder : nullptr;
  if (Tfix < 0) {
    a.stage("chunk_map");
    launch_chunk_map(a, st);
  }
  a.stage(a.saved ? "prep_save" : "prep");
  if (a.ncmax > 0) {
    if (a.saved)
      k_prep_bf<DK, true><<<dim3(a.ncmax, a.H), NTHR, 0, st>>>(
          q, k, a.g, bt, a.d, a.cmap, Tfix, a.H, a.Mq, a.Ms, a.Aq, a.As, a.QTp, a.Gw);
    else
      k_prep_bf<DK, false><<<dim3(a.ncmax, a.H), NTHR, 0, st>>>(
          q, k, a.g, bt, a.d, a.cmap, Tfix, a.H, a.Mq, a.Ms, a.Aq, a.As, nullptr, a.Gw);
  }
  if (a.segP > 1) {
    // Segmented forward for few long rows (fewer scan chains than the chip
    // has CUs): each row is cut into segP segments scanned side by side as
    // virtual rows of Tseq / segP tokens (chunk and token indices are those of
    // the real rows).  1. every segment's final state from a zero start and
    // its transition product (not of a row's last segment, which no later
    // segment needs); 2. the true state entering each segment
    // (k_seg_combine); 3. the output scan of every segment from that state
    // (with the chunk states for the backward in the training pair).
    // packed sequences: segments of each sequence from its table entry
    const SeqInfo* vsm = Tfix < 0 ? a.segmap : nullptr;
    const int Np = a.N * a.segP, Tp = Tfix < 0 ? -1 : a.Tseq / a.segP;
    if (Tfix < 0)
      k_seg_map<<<(Np + NTHR - 1) / NTHR, NTHR, 0, st>>>(a.smap, a.N, a.segP, a.segmap);
    seg_forward_states<DK, DV>(a, q, k, v, beta, bt, a.saved, vsm, Tp);
    a.stage(a.saved ? "scan_fwd_save" : "scan_fwd");
    float* htv = a.ht ? a.segHT : nullptr;
    if (a.saved)
      k_scan_fwd_bf<DK, DV, SCAN_BV, true, true><<<scan_blocks(Np, a.H, DV / SCAN_BV), NTHR, 0, st>>>(
          q, k, v, beta, bt, a.d, a.segX0, vsm, nullptr, Np, Tp, a.H, a.Mq, a.Ms, a.Aq, a.As,
          a.Gw, a.o, htv, a.Xq, a.Xs, a.Dq, a.Ds, nullptr, nullptr);
    else
      k_scan_fwd_bf<DK, DV, SCAN_BV, true, false><<<scan_blocks(Np, a.H, DV / SCAN_BV), NTHR, 0, st>>>(
          q, k, v, beta, bt, a.d, a.segX0, vsm, nullptr, Np, Tp, a.H, a.Mq, a.Ms, a.Aq, a.As,
          a.Gw, a.o, htv, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr);
    // the final state of each row is that of its last segment
    if (a.ht && seg_copy_rows<DK, DV>(a, a.ht, a.segHT, a.segP - 1) != hipSuccess)
      return hipErrorLaunchFailure;
    a.stage(nullptr);
    return hipGetLastError();
  }
  a.stage(a.saved ? "scan_fwd_save" : "scan_fwd");
  if (a.saved)
    k_scan_fwd_bf<DK, DV, SCAN_BV, true, true><<<scan_blocks(a.N, a.H, DV / SCAN_BV), NTHR, 0, st>>>(
        q, k, v, beta, bt, a.d, a.h0, a.smap, sord, a.N, Tfix, a.H, a.Mq, a.Ms, a.Aq, a.As, a.Gw, a.o, a.ht, a.Xq, a.Xs,
        a.Dq, a.Ds, a.Xfq, a.Xfs);
  else
    k_scan_fwd_bf<DK, DV, SCAN_BV, true, false><<<scan_blocks(a.N, a.H, DV / SCAN_BV), NTHR, 0, st>>>(
        q, k, v, beta, bt, a.d, a.h0, a.smap, sord, a.N, Tfix, a.H, a.Mq, a.Ms, a.Aq, a.As, a.Gw, a.o, a.ht, nullptr,
        nullptr, nullptr, nullptr, nullptr, nullptr);
  a.stage(nullptr);
  return hipGetLastError();
}

template <int DK, int DV>
static hipError_t run_bwd_bf(const LaunchArgs& a) {
  hipStream_t st = a.stream;
  const bf16_t* q = static_cast<const bf16_t*>(a.q);
  const bf16_t* k = static_cast<const bf16_t*>(a.k);
  const bf16_t* v = static_cast<const bf16_t*>(a.v);
  const bf16_t* beta = static_cast<const bf16_t*>(a.beta);
  const bf16_t* bt = static_cast<const bf16_t*>(a.beta_tilde);
  const bf16_t* dO = static_cast<const bf16_t*>(a.dO);
  if (a.N == 0) {
    k_reduce_dd<<<a.H, RDD_THR, 0, st>>>(a.ddp, 0, a.H, a.dd);
    return hipGetLastError();
  }
  // fixed-length rows need no tables (closed form in the kernels)
  const int Tfix = a.cu_seqlens ? -1 : a.Tseq;
  const int* sord = Tfix < 0 ? a.sorder : nullptr;
  if (a.segP > 1) {
    // Segmented backward (see run_fwd_bf): the forward's states as there
    // (the training pair's forward left them in the workspace, with the
    // transition products); then 1. every segment's state gradient at its
    // start from a zero end (not of a row's first segment); 2. the gradient of
    // the state leaving every segment (k_seg_combine_bwd, with Phi_p^T); 3. the
    // reverse scan of every segment from it, storing Y and dR for the
    // gradient kernel; dh0 is the first segment's.
    const int P = a.segP, Np = a.N * P, Nst = a.N * (P - 1);
    // packed sequences: segments of each sequence from its table entry (the
    // training pair's forward left the table in the workspace)
    const SeqInfo* vsm = Tfix < 0 ? a.segmap : nullptr;
    const int Tp = Tfix < 0 ? -1 : a.Tseq / P;
    if (!a.saved) {
      if (Tfix < 0) {
        a.stage("chunk_map");
        launch_chunk_map(a, st);
        k_seg_map<<<(Np + NTHR - 1) / NTHR, NTHR, 0, st>>>(a.smap, a.N, P, a.segmap);
      }
      a.stage("prep");
      if (a.ncmax > 0)
        k_prep_bf<DK, true><<<dim3(a.ncmax, a.H), NTHR, 0, st>>>(
            q, k, a.g, bt, a.d, a.cmap, Tfix, a.H, a.Mq, a.Ms, a.Aq, a.As, a.QTp, a.Gw);
      seg_forward_states<DK, DV>(a, q, k, v, beta, bt, true, vsm, Tp);
      a.stage("scan_fwd_store");
      k_scan_fwd_bf<DK, DV, SCAN_BV, false, true><<<scan_blocks(Np, a.H, DV / SCAN_BV), NTHR, 0, st>>>(
          q, k, v, beta, bt, a.d, a.segX0, vsm, nullptr, Np, Tp, a.H, a.Mq, a.Ms, a.Aq, a.As,
          a.Gw, nullptr, nullptr, a.Xq, a.Xs, a.Dq, a.Ds, nullptr, nullptr);
    }
    a.stage("scan_seg_grad");
    k_scan_bwd_bf<DK, DV, SCAN_BV, false><<<scan_blocks(Nst, a.H, DV / SCAN_BV), NTHR, 0, st>>>(
        q, k, dO, bt, a.d, nullptr, vsm, nullptr, Nst, Tp, a.H, a.Mq, a.Ms, a.Aq, a.As, a.QTp,
        a.Gw, a.segG, nullptr, nullptr, nullptr, nullptr, P, 1);
    a.stage("seg_combine_bwd");
    k_seg_combine_bwd<DK, DV><<<a.N * a.H * (DV / SEG_SL), NTHR, 0, st>>>(a.segPhi, a.segG, a.dht, P,
                                                                      a.H, a.segY0);
    a.stage("scan_bwd");
    k_scan_bwd_bf<DK, DV, SCAN_BV><<<scan_blocks(Np, a.H, DV / SCAN_BV), NTHR, 0, st>>>(
        q, k, dO, bt, a.d, a.segY0, vsm, nullptr, Np, Tp, a.H, a.Mq, a.Ms, a.Aq, a.As, a.QTp,
        a.Gw, a.dh0 ? a.segDH0 : nullptr, a.Yq, a.Ys, a.dRq, a.dRs);
    if (a.dh0 && seg_copy_rows<DK, DV>(a, a.dh0, a.segDH0, 0) != hipSuccess)
      return hipErrorLaunchFailure;
  } else if (!a.saved) {
    if (Tfix < 0) {
      a.stage("chunk_map");
      launch_chunk_map(a, st);
    }
    a.stage("prep");
    if (a.ncmax > 0)
      k_prep_bf<DK, true><<<dim3(a.ncmax, a.H), NTHR, 0, st>>>(
          q, k, a.g, bt, a.d, a.cmap, Tfix, a.H, a.Mq, a.Ms, a.Aq, a.As, a.QTp, a.Gw);
    // the chunk states (forward recurrence) and the reverse scan depend only on
    // prep's operands, not on each other (the reverse scan reads no state):
    // side by side, one workgroup of each per CU (68 + 92 KiB of LDS)
    a.stage("scans");
    side(
        st,
        [&](hipStream_t s1) {
          k_scan_fwd_bf<DK, DV, SCAN_BV, false, true><<<scan_blocks(a.N, a.H, DV / SCAN_BV), NTHR, 0, s1>>>(
              q, k, v, beta, bt, a.d, a.h0, a.smap, sord, a.N, Tfix, a.H, a.Mq, a.Ms, a.Aq, a.As, a.Gw, nullptr,
              nullptr, a.Xq, a.Xs, a.Dq, a.Ds, a.Xfq, a.Xfs);
        },
        [&](hipStream_t s2) {
          k_scan_bwd_bf<DK, DV, SCAN_BV><<<scan_blocks(a.N, a.H, DV / SCAN_BV), NTHR, 0, s2>>>(
              q, k, dO, bt, a.d, a.dht, a.smap, sord, a.N, Tfix, a.H, a.Mq, a.Ms, a.Aq, a.As, a.QTp, a.Gw, a.dh0,
              a.Yq, a.Ys, a.dRq, a.dRs);
        });
  }
  if (a.segP <= 1 && a.saved) {
    a.stage("scan_bwd");
    k_scan_bwd_bf<DK, DV, SCAN_BV><<<scan_blocks(a.N, a.H, DV / SCAN_BV), NTHR, 0, st>>>(
        q, k, dO, bt, a.d, a.dht, a.smap, sord, a.N, Tfix, a.H, a.Mq, a.Ms, a.Aq, a.As, a.QTp, a.Gw, a.dh0, a.Yq,
        a.Ys, a.dRq, a.dRs);
  }
  a.stage("intra_bwd");
  if constexpr (DK > 128 || DV > 128) {
    // head dim 256: passes of 128 dk columns, one workgroup per chunk-head (at
    // dv = 256 the persistent kernel spills; this one is 25% faster there)
    if (a.ncmax > 0)
      k_intra_bwd_wide<DK, DV><<<dim3(a.ncmax, a.H), IB_THR, 0, st>>>(
          q, k, v, dO, beta, bt, a.d, a.cmap, Tfix, a.H, a.Gw, a.Xq, a.Xs, a.Dq, a.Ds, a.Yq, a.Ys,
          a.dRq, a.dRs, a.dq, a.dk_, a.dv_, a.dbeta, a.dbeta_tilde, a.dg, a.ddp);
  } else {
    if (a.ncmax > 0)
      k_intra_bwd_bf<DK, DV><<<dim3(intra_bwd_grid((long)a.ncmax * a.H)), IB_THR, 0, st>>>(
          q, k, v, dO, beta, bt, a.d, a.cmap, Tfix, a.H, a.Gw, a.Xq, a.Xs, a.Dq, a.Ds, a.Yq, a.Ys, a.dRq,
          a.dRs, a.ncmax, a.dq, a.dk_, a.dv_, a.dbeta, a.dbeta_tilde, a.dg, a.ddp);
  }
  a.stage("reduce_dd");
  k_reduce_dd<<<a.H, RDD_THR, 0, st>>>(a.ddp, a.ncmax, a.H, a.dd);
  a.stage(nullptr);
  return hipGetLastError();
}

template <bool BWD>
static hipError_t dispatch_bf(const LaunchArgs& a) {
  if (a.dk == 64 && a.dv == 64) return BWD ? run_bwd_bf<64, 64>(a) : run_fwd_bf<64, 64>(a);
  if (a.dk == 128 && a.dv == 128) return BWD ? run_bwd_bf<128, 128>(a) : run_fwd_bf<128, 128>(a);
  if (a.dk == 64 && a.dv == 128) return BWD ? run_bwd_bf<64, 128>(a) : run_fwd_bf<64, 128>(a);
  if (a.dk == 128 && a.dv == 64) return BWD ? run_bwd_bf<128, 64>(a) : run_fwd_bf<128, 64>(a);
  // head dim 256 (the paper's models)
  if (a.dk == 256 && a.dv == 256) return BWD ? run_bwd_bf<256, 256>(a) : run_fwd_bf<256, 256>(a);
  if (a.dk == 128 && a.dv == 256) return BWD ? run_bwd_bf<128, 256>(a) : run_fwd_bf<128, 256>(a);
  if (a.dk == 256 && a.dv == 128) return BWD ? run_bwd_bf<256, 128>(a) : run_fwd_bf<256, 128>(a);
  return hipErrorInvalidValue;
}

template <bool BWD, typename Tin>
static hipError_t dispatch_dims(const LaunchArgs& a) {
  if (a.dk == 64 && a.dv == 64) return BWD ? run_bwd<Tin, 64, 64>(a) : run_fwd<Tin, 64, 64>(a);
  return hipErrorInvalidValue;
}

hipError_t launch_fwd(const LaunchArgs& a) {
  return a.bf16 ? dispatch_bf<false>(a) : dispatch_dims<false, float>(a);
}

hipError_t launch_bwd(const LaunchArgs& a) {
  return a.bf16 ? dispatch_bf<true>(a) : dispatch_dims<true, float>(a);
}

}  // namespace comba
