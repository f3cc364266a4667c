// Host side of the C ABI declared in include/comba.h: argument validation,
// workspace layout and kernel sequencing on the caller's stream.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdlib.h>

#include <string>
#include <vector>

#include "comba.h"
#include "comba_launch.h"

namespace {

constexpr int kChunk = 64;
constexpr size_t kAlign = 256;

size_t round_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Dims {
  bool bf16, packed;
  int dk, dv, H, N, Tseq, Ttot, ncmax;
  int maxch;  // chunks of the longest sequence (packed: 0 without the host offsets)
};

// Validates the shape; fills dims on success.  `wide` also admits head dim 256
// (bf16 inputs, with 128 or 256 on the other side).
comba_status check_shape(const comba_shape* s, Dims* out, bool wide = false) {
  if (!s) return COMBA_ERR_NULL;
  if (s->in_dtype != COMBA_F32 && s->in_dtype != COMBA_BF16) return COMBA_ERR_DTYPE;
  const bool bf16 = s->in_dtype == COMBA_BF16;
  if (s->chunk != kChunk) return COMBA_ERR_SHAPE;
  if (s->B < 0 || s->T < 0 || s->H <= 0 || s->H > 65535) return COMBA_ERR_SHAPE;
  const bool dk_ok = s->dk == 64 || (bf16 && s->dk == 128);
  const bool dv_ok = s->dv == 64 || (bf16 && s->dv == 128);
  const bool big = bf16 && wide && (s->dk == 256 || s->dv == 256) &&
                   (s->dk == 128 || s->dk == 256) && (s->dv == 128 || s->dv == 256);
  if (!big && (!dk_ok || !dv_ok)) return COMBA_ERR_SHAPE;
  Dims d;
  d.bf16 = bf16;
  d.packed = s->cu_seqlens != nullptr;
  d.dk = s->dk;
  d.dv = s->dv;
  d.H = s->H;
  if (s->cu_seqlens) {
    if (s->B != 1 || s->num_seqs < 0) return COMBA_ERR_SHAPE;
    d.N = s->num_seqs;
    d.Tseq = 0;
    d.maxch = 0;
    if (s->cu_seqlens_host) {
      // the host copy of the offsets: 0 = cu[0] <= cu[1] <= ... <= cu[N] = T
      const int32_t* cu = s->cu_seqlens_host;
      if (cu[0] != 0 || cu[d.N] != s->T) return COMBA_ERR_SHAPE;
      for (int i = 0; i < d.N; ++i) {
        if (cu[i + 1] < cu[i]) return COMBA_ERR_SHAPE;
        const int nch = (cu[i + 1] - cu[i] + kChunk - 1) / kChunk;
        if (nch > d.maxch) d.maxch = nch;
      }
    }
  } else {
    if (s->cu_seqlens_host) return COMBA_ERR_SHAPE;  // offsets without a packed batch
    if (s->num_seqs != s->B) return COMBA_ERR_SHAPE;
    d.N = s->B;
    d.Tseq = s->T;
    d.maxch = (s->T + kChunk - 1) / kChunk;
  }
  const int64_t ttot = s->cu_seqlens ? (int64_t)s->T : (int64_t)s->B * s->T;
  if (ttot > INT32_MAX / 2) return COMBA_ERR_SHAPE;
  if (d.N > 65535 * 1024) return COMBA_ERR_SHAPE;
  // the scans run one workgroup per (sequence, head, 32-column slice) in a 1-D grid
  if ((int64_t)d.N * d.H * 8 > INT32_MAX) return COMBA_ERR_SHAPE;
  d.Ttot = (int)ttot;
  // fixed-length rows: ceil(T / 64) chunks each; packed sequences: each
  // sequence adds at most one partial chunk to ceil(Ttot / 64)
  const int64_t nc = s->cu_seqlens ? (ttot + kChunk - 1) / kChunk + d.N
                                   : (int64_t)d.N * ((d.Tseq + kChunk - 1) / kChunk);
  if (nc > INT32_MAX / 2) return COMBA_ERR_SHAPE;
  d.ncmax = (int)nc;
  *out = d;
  return COMBA_OK;
}

// Shape rules of the token-by-token entry point: those of check_shape, except
// that the chunk length is not used and dk, dv may each be 64, 128 or 256 for
// either input dtype (pairs with 64 and 256 excepted).
comba_status check_shape_recurrent(const comba_shape* s, Dims* out) {
  if (!s) return COMBA_ERR_NULL;
  comba_shape c = *s;
  c.chunk = kChunk;
  const bool f32 = c.in_dtype == COMBA_F32;
  if (f32) c.in_dtype = COMBA_BF16;  // the head-size rule of the bf16 path
  const bool wide = c.dk == 256 || c.dv == 256;
  if (wide) {
    if ((c.dk != 128 && c.dk != 256) || (c.dv != 128 && c.dv != 256)) return COMBA_ERR_SHAPE;
    c.dk = c.dv = 128;  // checked as d = 128, restored below
  }
  const comba_status st = check_shape(&c, out);
  if (st == COMBA_OK) {
    out->bf16 = !f32;
    out->dk = s->dk;
    out->dv = s->dv;
  }
  return st;
}

// Segments of the stateless bf16 forward (comba::LaunchArgs::segP; 1 = off).
// Rows of fixed length are cut when their scan has at most half as many chains
// (N H dv / 32) as the device has CUs, into the largest power of two P for
// which the segments' chains are at most two per CU, P divides the row's
// chunks and every segment keeps at least 16 chunks.  COMBA_SCAN_SEGMENTS overrides the
// choice: 1 disables, P >= 2 forces P when it divides the row's chunks (P <= 64;
// any other P disables); unset or 0 keeps the automatic choice.
int seg_parts(const Dims& d) {
  if (!d.bf16 || d.N <= 0) return 1;
  // fixed-length rows: whole chunks, P dividing them; packed sequences: any P
  // (a sequence's segments are ceil(n / P) chunks, the last ones shorter or
  // empty), chosen automatically only when the host offsets give the lengths
  const bool packed = d.packed;
  if (!packed && (d.Tseq <= 0 || d.Tseq % kChunk)) return 1;
  const int n = packed ? d.maxch : d.Tseq / kChunk;
  if (const char* env = getenv("COMBA_SCAN_SEGMENTS")) {
    const int P = atoi(env);  // 0 (or not a number): the automatic choice below
    if (P != 0) return P >= 2 && P <= 64 && (packed || n % P == 0) ? P : 1;
  }
  if (n <= 0) return 1;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 1;
  const long chains = (long)d.N * d.H * (d.dv / 32);
  if (cus <= 0 || 2 * chains > cus) return 1;
  int P = 1;
  while (P < 64 && chains * 2 * P <= 2L * cus && (packed || n % (2 * P) == 0) && n / (2 * P) >= 16)
    P *= 2;
  return P;
}

struct Layout {
  size_t cmap, smap, sord, M, A, G, X, D, Y, dR, ddp, QT, Xfin, total;
  size_t segF, segPhi, segX0, segHT, segG, segY0, segDH0, segmap;  // segmented scans (segP > 1)
  size_t Xs, Ds, Ys, dRs, Xfs;  // bf16 path: scales of the int16 X, D, Y, dR, final-state sink
  size_t Ms, As;                // bf16 path: row scales of M, column scales of A
};

Layout layout(const Dims& d, bool bwd, int segP = 1) {
  Layout L{};
  const size_t chh = (size_t)d.ncmax * d.H;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += round_up(bytes);
    return at;
  };
  L.cmap = take((size_t)d.ncmax * sizeof(comba::ChunkInfo));
  L.smap = take((size_t)(d.N > 0 ? d.N : 1) * sizeof(comba::SeqInfo));
  L.sord = take((size_t)(d.N > 0 ? d.N : 1) * sizeof(int));
  L.G = take(chh * kChunk * sizeof(float));
  if (d.bf16) {
    // bf16 path: M, A as int16 with row (M) and column (A) scales; the
    // backward also keeps Q^T
    L.M = take(chh * kChunk * kChunk * sizeof(int16_t));
    L.Ms = take(chh * kChunk * sizeof(float));
    L.A = take(chh * kChunk * kChunk * sizeof(int16_t));
    L.As = take(chh * kChunk * sizeof(float));
    if (bwd) {
      // Q^T; X, D, Y, dR as int16 + one fp32 scale per 32 values
      const size_t nf = (size_t)(d.N > 0 ? d.N : 1) * d.H;
      const size_t nb = d.dv / 32;
      L.QT = take(chh * d.dk * kChunk * sizeof(uint16_t));
      L.Xfin = take(nf * d.dk * d.dv * sizeof(int16_t));
      L.Xfs = take(nf * d.dk * nb * sizeof(float));
      L.X = take(chh * d.dk * d.dv * sizeof(int16_t));
      L.Xs = take(chh * d.dk * nb * sizeof(float));
      L.D = take(chh * kChunk * d.dv * sizeof(int16_t));
      L.Ds = take(chh * kChunk * nb * sizeof(float));
      L.Y = take(chh * d.dk * d.dv * sizeof(int16_t));
      L.Ys = take(chh * d.dk * nb * sizeof(float));
      L.dR = take(chh * kChunk * d.dv * sizeof(int16_t));
      L.dRs = take(chh * kChunk * nb * sizeof(float));
      L.ddp = take(chh * sizeof(float));
    }
  } else {
    L.M = take(chh * kChunk * kChunk * sizeof(float));
    L.A = take(chh * kChunk * kChunk * sizeof(float));
  }
  if (!d.bf16 && bwd) {
    L.X = take(chh * d.dk * d.dv * sizeof(float));
    L.D = take(chh * kChunk * d.dv * sizeof(float));
    L.Y = take(chh * d.dk * d.dv * sizeof(float));
    L.dR = take(chh * kChunk * d.dv * sizeof(float));
    L.ddp = take(chh * sizeof(float));
  }
  if (segP > 1) {
    // per virtual row (segment) and head, fp32: F, X0, HT (dk x dv), Phi (dk x
    // dk); the backward-sized workspace (training pair, stateless backward)
    // also G, Y0, DH0 (dk x dv)
    const size_t nvr = (size_t)d.N * segP * d.H;
    L.segmap = take((size_t)d.N * segP * sizeof(comba::SeqInfo));  // packed: virtual rows
    L.segF = take(nvr * d.dk * d.dv * sizeof(float));
    L.segPhi = take(nvr * d.dk * d.dk * sizeof(float));
    L.segX0 = take(nvr * d.dk * d.dv * sizeof(float));
    L.segHT = take(nvr * d.dk * d.dv * sizeof(float));
    if (bwd) {
      L.segG = take(nvr * d.dk * d.dv * sizeof(float));
      L.segY0 = take(nvr * d.dk * d.dv * sizeof(float));
      L.segDH0 = take(nvr * d.dk * d.dv * sizeof(float));
    }
  }
  L.total = off;
  return L;
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

// Per-thread stage timing (comba_profile_enable / comba_profile_read).  A
// session records, for every call, one event before each kernel stage and one
// after the last; events come from a pool that is created on demand and
// reused by later sessions.
constexpr size_t kMaxEvents = 4096;
constexpr size_t kMaxMarksPerCall = 16;
struct Profile {
  bool on = false;
  size_t n = 0;
  std::vector<hipEvent_t> ev;
  std::vector<const char*> names;
  std::string only;   // when not empty: record only this stage (its start and its end)
  bool open = false;  // the selected stage's start is recorded, its end comes next
};
thread_local Profile g_prof;

void prof_mark(void* ctx, hipStream_t st, const char* name) {
  Profile* p = static_cast<Profile*>(ctx);
  if (!p->only.empty()) {
    const bool sel = name && p->only == name;
    if (!sel && !p->open) return;  // neither the selected stage's start nor its end
    if (!sel) name = nullptr;      // the selected stage's end: no stage of its own
    p->open = sel;
  }
  if (p->n == p->ev.size()) {
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return;
    p->ev.push_back(e);
    p->names.push_back(nullptr);
  }
  if (hipEventRecord(p->ev[p->n], st) != hipSuccess) return;
  p->names[p->n] = name;
  ++p->n;
}

template <typename Args>
void attach_profile(Args& a) {
  // a call records at most kMaxMarksPerCall marks; stop at the pool limit so
  // that no call is recorded partially
  if (!g_prof.on || g_prof.n + kMaxMarksPerCall > kMaxEvents) return;
  a.hook.mark = prof_mark;
  a.hook.ctx = &g_prof;
}

void carve(comba::LaunchArgs& a, const Layout& L, void* ws, bool bwd, int segP = 1) {
  char* base = static_cast<char*>(ws);
  a.segP = segP;
  if (segP > 1) {
    a.segmap = reinterpret_cast<comba::SeqInfo*>(base + L.segmap);
    a.segF = reinterpret_cast<float*>(base + L.segF);
    a.segPhi = reinterpret_cast<float*>(base + L.segPhi);
    a.segX0 = reinterpret_cast<float*>(base + L.segX0);
    a.segHT = reinterpret_cast<float*>(base + L.segHT);
    if (bwd) {
      a.segG = reinterpret_cast<float*>(base + L.segG);
      a.segY0 = reinterpret_cast<float*>(base + L.segY0);
      a.segDH0 = reinterpret_cast<float*>(base + L.segDH0);
    }
  }
  a.cmap = reinterpret_cast<comba::ChunkInfo*>(base + L.cmap);
  a.smap = reinterpret_cast<comba::SeqInfo*>(base + L.smap);
  a.sorder = reinterpret_cast<int*>(base + L.sord);
  a.Mw = reinterpret_cast<float*>(base + L.M);
  a.Aw = reinterpret_cast<float*>(base + L.A);
  a.Gw = reinterpret_cast<float*>(base + L.G);
  if (a.bf16) {
    a.Mq = reinterpret_cast<int16_t*>(base + L.M);
    a.Ms = reinterpret_cast<float*>(base + L.Ms);
    a.Aq = reinterpret_cast<int16_t*>(base + L.A);
    a.As = reinterpret_cast<float*>(base + L.As);
    if (bwd) a.QTp = reinterpret_cast<uint16_t*>(base + L.QT);
  }
  if (bwd && a.bf16) {
    a.Xfq = reinterpret_cast<int16_t*>(base + L.Xfin);
    a.Xfs = reinterpret_cast<float*>(base + L.Xfs);
    a.Xq = reinterpret_cast<int16_t*>(base + L.X);
    a.Xs = reinterpret_cast<float*>(base + L.Xs);
    a.Dq = reinterpret_cast<int16_t*>(base + L.D);
    a.Ds = reinterpret_cast<float*>(base + L.Ds);
    a.Yq = reinterpret_cast<int16_t*>(base + L.Y);
    a.Ys = reinterpret_cast<float*>(base + L.Ys);
    a.dRq = reinterpret_cast<int16_t*>(base + L.dR);
    a.dRs = reinterpret_cast<float*>(base + L.dRs);
    a.ddp = reinterpret_cast<float*>(base + L.ddp);
  } else if (bwd) {
    a.Xw = reinterpret_cast<float*>(base + L.X);
    a.Dw = reinterpret_cast<float*>(base + L.D);
    a.Yw = reinterpret_cast<float*>(base + L.Y);
    a.dRw = reinterpret_cast<float*>(base + L.dR);
    a.ddp = reinterpret_cast<float*>(base + L.ddp);
  }
}

void fill_common(comba::LaunchArgs& a, const Dims& d, const comba_shape* s) {
  a.bf16 = d.bf16;
  a.dk = d.dk;
  a.dv = d.dv;
  a.H = d.H;
  a.N = d.N;
  a.Tseq = d.Tseq;
  a.Ttot = d.Ttot;
  a.ncmax = d.ncmax;
  a.cu_seqlens = s->cu_seqlens;
}

comba_status chunk_fwd(bool save, const comba_shape* shape, const void* q, const void* k,
                       const void* v, const float* g, const void* beta, const void* beta_tilde,
                       const float* d, const float* h0, float* o, float* ht, void* ws,
                       size_t ws_bytes, void* stream) {
  Dims dm;
  comba_status st = check_shape(shape, &dm, true);
  if (st != COMBA_OK) return st;
  // token tensors may be NULL when the call has no tokens (states pass through)
  const bool tok = dm.Ttot > 0;
  if ((tok && (!q || !k || !v || !g || !beta || !o)) || !d || !ws) return COMBA_ERR_NULL;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(ws, kAlign) ||
      !aligned(g, 4) || !aligned(d, 4) || !aligned(o, 16) || (h0 && !aligned(h0, 16)) ||
      (ht && !aligned(ht, 16)) || !aligned(beta, dm.bf16 ? 2 : 4) ||
      !aligned(beta_tilde, dm.bf16 ? 2 : 4))
    return COMBA_ERR_ALIGN;
  // the segmented scan when the workspace holds its buffers (sized by
  // comba_fwd_workspace_bytes / comba_bwd_workspace_bytes), else the plain one
  int segP = seg_parts(dm);
  Layout L = layout(dm, save, segP);
  if (ws_bytes < L.total && segP > 1) {
    segP = 1;
    L = layout(dm, save, 1);
  }
  if (ws_bytes < L.total) return COMBA_ERR_WORKSPACE;
  comba::LaunchArgs a{};
  fill_common(a, dm, shape);
  a.saved = save;
  a.q = q;
  a.k = k;
  a.v = v;
  a.beta = beta;
  a.beta_tilde = beta_tilde ? beta_tilde : beta;  // NULL: tied to beta
  a.g = g;
  a.d = d;
  a.h0 = h0;
  a.o = o;
  a.ht = ht;
  a.stream = static_cast<hipStream_t>(stream);
  carve(a, L, ws, save, segP);
  attach_profile(a);
  if (dm.N == 0) return COMBA_OK;
  return comba::launch_fwd(a) == hipSuccess ? COMBA_OK : COMBA_ERR_HIP;
}

comba_status chunk_bwd(bool saved, const comba_shape* shape, const void* q, const void* k,
                       const void* v, const float* g, const void* beta, const void* beta_tilde,
                       const float* d, const float* h0, const void* dO, const float* dht,
                       float* dq, float* dk, float* dv, float* dg, float* dbeta,
                       float* dbeta_tilde, float* dd, float* dh0, void* ws, size_t ws_bytes,
                       void* stream) {
  Dims dm;
  comba_status st = check_shape(shape, &dm, true);
  if (st != COMBA_OK) return st;
  // token tensors may be NULL when the call has no tokens (states pass through)
  const bool tok = dm.Ttot > 0;
  // a separate beta~ needs its own gradient
  if ((tok && (!q || !k || !v || !g || !beta || !dO || !dq || !dk || !dv || !dg || !dbeta ||
               (beta_tilde && !dbeta_tilde))) ||
      !d || !dd || !ws)
    return COMBA_ERR_NULL;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(dO, 16) ||
      !aligned(ws, kAlign) || !aligned(g, 4) || !aligned(d, 4) || !aligned(dq, 16) ||
      !aligned(dk, 16) || !aligned(dv, 16) || !aligned(dg, 4) || !aligned(dbeta, 4) ||
      !aligned(dd, 4) || (h0 && !aligned(h0, 16)) || (dht && !aligned(dht, 16)) ||
      (dh0 && !aligned(dh0, 16)) || !aligned(beta, dm.bf16 ? 2 : 4) ||
      !aligned(beta_tilde, dm.bf16 ? 2 : 4) || !aligned(dbeta_tilde, 4))
    return COMBA_ERR_ALIGN;
  // segmented as the forward of the pair was (the same shape, device and
  // COMBA_SCAN_SEGMENTS give the same choice and the same workspace layout)
  int segP = seg_parts(dm);
  Layout L = layout(dm, true, segP);
  if (ws_bytes < L.total && segP > 1) {
    segP = 1;
    L = layout(dm, true, 1);
  }
  if (ws_bytes < L.total) return COMBA_ERR_WORKSPACE;
  comba::LaunchArgs a{};
  fill_common(a, dm, shape);
  a.saved = saved;
  a.q = q;
  a.k = k;
  a.v = v;
  a.beta = beta;
  a.beta_tilde = beta_tilde ? beta_tilde : beta;  // NULL: tied to beta
  a.dO = dO;
  a.g = g;
  a.d = d;
  a.h0 = h0;
  a.dht = dht;
  a.dq = dq;
  a.dk_ = dk;
  a.dv_ = dv;
  a.dg = dg;
  a.dbeta = dbeta;
  a.dbeta_tilde = dbeta_tilde;  // NULL: dbeta holds the total derivative
  a.dd = dd;
  a.dh0 = dh0;
  a.stream = static_cast<hipStream_t>(stream);
  carve(a, L, ws, true, segP);
  attach_profile(a);
  return comba::launch_bwd(a) == hipSuccess ? COMBA_OK : COMBA_ERR_HIP;
}

comba_status recurrent_fwd(const comba_shape* shape, const void* q, const void* k, const void* v,
                           const float* g, const void* beta, const void* beta_tilde,
                           const float* d, const float* h0, float* o, float* ht, void* stream) {
  Dims dm;
  comba_status st = check_shape_recurrent(shape, &dm);
  if (st != COMBA_OK) return st;
  const bool tok = dm.Ttot > 0;
  if ((tok && (!q || !k || !v || !g || !beta || !o)) || !d) return COMBA_ERR_NULL;
  const size_t eb = dm.bf16 ? 2 : 4;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(g, 4) ||
      !aligned(d, 4) || !aligned(o, 16) || (h0 && !aligned(h0, 16)) || (ht && !aligned(ht, 16)) ||
      !aligned(beta, eb) || !aligned(beta_tilde, eb))
    return COMBA_ERR_ALIGN;
  comba::RecurrentArgs a{};
  a.bf16 = dm.bf16;
  a.dk = dm.dk;
  a.dv = dm.dv;
  a.H = dm.H;
  a.N = dm.N;
  a.Tseq = dm.Tseq;
  a.Ttot = dm.Ttot;
  a.cu_seqlens = shape->cu_seqlens;
  a.q = q;
  a.k = k;
  a.v = v;
  a.beta = beta;
  a.beta_tilde = beta_tilde ? beta_tilde : beta;  // NULL: tied to beta
  a.g = g;
  a.d = d;
  a.h0 = h0;
  a.o = o;
  a.ht = ht;
  a.stream = static_cast<hipStream_t>(stream);
  attach_profile(a);
  return comba::launch_recurrent(a) == hipSuccess ? COMBA_OK : COMBA_ERR_HIP;
}

// Prologue: 64-token runs of the packed token axis and the per-run dw partials.
constexpr int kRun = 64;
constexpr float kPrologueEps = 1e-6f;

size_t prologue_ws_bytes(const Dims& d) {
  const size_t nruns = ((size_t)d.Ttot + kRun - 1) / kRun;
  return round_up(nruns * d.H * (2 * d.dk + d.dv) * 4 * sizeof(float)) + kAlign;
}

comba_status prologue(bool bwd, const comba_shape* shape, const void* xq, const void* xk,
                      const void* xv, const float* wq, const float* wk, const float* wv, void* q,
                      void* k, void* v, const float* gq, const float* gk, const float* gv,
                      float* dxq, float* dxk, float* dxv, float* dwq, float* dwk, float* dwv,
                      void* ws, size_t ws_bytes, void* stream) {
  Dims dm;
  comba_status st = check_shape_recurrent(shape, &dm);
  if (st != COMBA_OK) return st;
  const bool tok = dm.Ttot > 0;
  if (tok && dm.N == 0) return COMBA_ERR_SHAPE;  // tokens must belong to a sequence
  if (tok && (!xq || !xk || !xv || !wq || !wk || !wv)) return COMBA_ERR_NULL;
  if (!bwd && tok && (!q || !k || !v)) return COMBA_ERR_NULL;
  if (bwd && ((tok && (!gq || !gk || !gv || !dxq || !dxk || !dxv)) || !dwq || !dwk || !dwv || !ws))
    return COMBA_ERR_NULL;
  if (!aligned(xq, 16) || !aligned(xk, 16) || !aligned(xv, 16) || !aligned(wq, 4) ||
      !aligned(wk, 4) || !aligned(wv, 4) || !aligned(q, 16) || !aligned(k, 16) ||
      !aligned(v, 16) || !aligned(gq, 16) || !aligned(gk, 16) || !aligned(gv, 16) ||
      !aligned(dxq, 16) || !aligned(dxk, 16) || !aligned(dxv, 16) || !aligned(dwq, 4) ||
      !aligned(dwk, 4) || !aligned(dwv, 4) || !aligned(ws, kAlign))
    return COMBA_ERR_ALIGN;
  if (bwd && ws_bytes < prologue_ws_bytes(dm)) return COMBA_ERR_WORKSPACE;
  comba::PrologueArgs a{};
  a.bf16 = dm.bf16;
  a.dk = dm.dk;
  a.dv = dm.dv;
  a.H = dm.H;
  a.N = dm.N;
  a.Tseq = dm.Tseq;
  a.Ttot = dm.Ttot;
  a.nruns = (dm.Ttot + kRun - 1) / kRun;
  a.eps = kPrologueEps;
  a.cu_seqlens = shape->cu_seqlens;
  a.xq = xq;
  a.xk = xk;
  a.xv = xv;
  a.wq = wq;
  a.wk = wk;
  a.wv = wv;
  a.q = q;
  a.k = k;
  a.v = v;
  a.gq = gq;
  a.gk = gk;
  a.gv = gv;
  a.dxq = dxq;
  a.dxk = dxk;
  a.dxv = dxv;
  a.dwq = dwq;
  a.dwk = dwk;
  a.dwv = dwv;
  if (bwd) {
    const size_t nr = (size_t)a.nruns * a.H;
    float* base = static_cast<float*>(ws);
    a.dwpq = base;
    a.dwpk = base + nr * a.dk * 4;
    a.dwpv = base + 2 * nr * a.dk * 4;
  }
  a.stream = static_cast<hipStream_t>(stream);
  attach_profile(a);
  return comba::launch_prologue(a, bwd) == hipSuccess ? COMBA_OK : COMBA_ERR_HIP;
}

comba_status gate(const comba_shape* shape, const float* o, const void* z, void* y,
                  const float* dy, float* dout, float* dz, void* stream) {
  Dims dm;
  comba_status st = check_shape_recurrent(shape, &dm);
  if (st != COMBA_OK) return st;
  const long n = (long)dm.Ttot * dm.H * dm.dv;
  if (n > 0 && (!o || !z || (dy ? (!dout || !dz) : !y))) return COMBA_ERR_NULL;
  if (!aligned(o, 16) || !aligned(z, 16) || !aligned(y, 16) || !aligned(dy, 16) ||
      !aligned(dout, 16) || !aligned(dz, 16))
    return COMBA_ERR_ALIGN;
  return comba::launch_gate(dm.bf16, n, o, z, y, dy, dout, dz, static_cast<hipStream_t>(stream)) ==
                 hipSuccess
             ? COMBA_OK
             : COMBA_ERR_HIP;
}

}  // namespace

namespace comba {
// The stateless forward's workspace without the segmented scan's buffers: a
// call given this much runs the plain scan (comba_chunk_fwd_noalloc).
size_t fwd_workspace_bytes_plain(const comba_shape* shape) {
  Dims d;
  if (check_shape(shape, &d, true) != COMBA_OK) return 0;
  return layout(d, false, 1).total;
}
}  // namespace comba

extern "C" {

comba_status comba_gate_fwd(const comba_shape* shape, const float* o, const void* z, void* y,
                            void* stream) {
  return gate(shape, o, z, y, nullptr, nullptr, nullptr, stream);
}

comba_status comba_gate_bwd(const comba_shape* shape, const float* o, const void* z,
                            const float* dy, float* dout, float* dz, void* stream) {
  if (!dy && shape) {
    Dims dm;
    if (check_shape_recurrent(shape, &dm) == COMBA_OK && dm.Ttot > 0) return COMBA_ERR_NULL;
  }
  return gate(shape, o, z, nullptr, dy, dout, dz, stream);
}

size_t comba_prologue_workspace_bytes(const comba_shape* shape) {
  Dims d;
  if (check_shape_recurrent(shape, &d) != COMBA_OK) return 0;
  return prologue_ws_bytes(d);
}

comba_status comba_prologue_fwd(const comba_shape* shape, const void* xq, const void* xk,
                                const void* xv, const float* wq, const float* wk, const float* wv,
                                void* q, void* k, void* v, void* stream) {
  return prologue(false, shape, xq, xk, xv, wq, wk, wv, q, k, v, nullptr, nullptr, nullptr,
                  nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 0, stream);
}

comba_status comba_prologue_bwd(const comba_shape* shape, const void* xq, const void* xk,
                                const void* xv, const float* wq, const float* wk, const float* wv,
                                const float* gq, const float* gk, const float* gv, float* dxq,
                                float* dxk, float* dxv, float* dwq, float* dwk, float* dwv,
                                void* ws, size_t ws_bytes, void* stream) {
  return prologue(true, shape, xq, xk, xv, wq, wk, wv, nullptr, nullptr, nullptr, gq, gk, gv, dxq,
                  dxk, dxv, dwq, dwk, dwv, ws, ws_bytes, stream);
}

size_t comba_fwd_workspace_bytes(const comba_shape* shape) {
  Dims d;
  if (check_shape(shape, &d, true) != COMBA_OK) return 0;
  return layout(d, false, seg_parts(d)).total;
}

size_t comba_bwd_workspace_bytes(const comba_shape* shape) {
  Dims d;
  if (check_shape(shape, &d, true) != COMBA_OK) return 0;
  return layout(d, true, seg_parts(d)).total;
}

comba_status comba_profile_enable(int enable) {
  g_prof.on = enable != 0;
  g_prof.n = 0;
  g_prof.open = false;
  return COMBA_OK;
}

comba_status comba_profile_select(const char* stage) {
  g_prof.only = stage ? stage : "";
  g_prof.open = false;
  return COMBA_OK;
}

int comba_profile_read(float* ms, const char** names, int capacity) {
  if (g_prof.n < 2) return 0;
  if (hipEventSynchronize(g_prof.ev[g_prof.n - 1]) != hipSuccess) return -1;
  int out = 0;
  for (size_t i = 0; i + 1 < g_prof.n && out < capacity; ++i) {
    if (!g_prof.names[i]) continue;  // end-of-call mark
    float t = 0.f;
    if (hipEventElapsedTime(&t, g_prof.ev[i], g_prof.ev[i + 1]) != hipSuccess) return -1;
    if (ms) ms[out] = t;
    if (names) names[out] = g_prof.names[i];
    ++out;
  }
  return out;
}

comba_status comba_chunk_fwd(const comba_shape* shape, const void* q, const void* k, const void* v,
                             const float* g, const void* beta, const void* beta_tilde,
                             const float* d, const float* h0, float* o, float* ht, void* ws,
                             size_t ws_bytes, void* stream) {
  return chunk_fwd(false, shape, q, k, v, g, beta, beta_tilde, d, h0, o, ht, ws, ws_bytes, stream);
}

comba_status comba_chunk_fwd_save(const comba_shape* shape, const void* q, const void* k,
                                  const void* v, const float* g, const void* beta,
                                  const void* beta_tilde, const float* d, const float* h0, float* o,
                                  float* ht, void* ws, size_t ws_bytes, void* stream) {
  return chunk_fwd(true, shape, q, k, v, g, beta, beta_tilde, d, h0, o, ht, ws, ws_bytes, stream);
}

comba_status comba_chunk_bwd(const comba_shape* shape, const void* q, const void* k, const void* v,
                             const float* g, const void* beta, const void* beta_tilde,
                             const float* d, const float* h0, const void* dO, const float* dht,
                             float* dq, float* dk, float* dv, float* dg, float* dbeta,
                             float* dbeta_tilde, float* dd, float* dh0, void* ws, size_t ws_bytes,
                             void* stream) {
  return chunk_bwd(false, shape, q, k, v, g, beta, beta_tilde, d, h0, dO, dht, dq, dk, dv, dg,
                   dbeta, dbeta_tilde, dd, dh0, ws, ws_bytes, stream);
}

comba_status comba_chunk_bwd_saved(const comba_shape* shape, const void* q, const void* k,
                                   const void* v, const float* g, const void* beta,
                                   const void* beta_tilde, const float* d, const float* h0,
                                   const void* dO, const float* dht, float* dq, float* dk,
                                   float* dv, float* dg, float* dbeta, float* dbeta_tilde,
                                   float* dd, float* dh0, void* ws, size_t ws_bytes,
                                   void* stream) {
  return chunk_bwd(true, shape, q, k, v, g, beta, beta_tilde, d, h0, dO, dht, dq, dk, dv, dg,
                   dbeta, dbeta_tilde, dd, dh0, ws, ws_bytes, stream);
}

comba_status comba_recurrent_fwd(const comba_shape* shape, const void* q, const void* k,
                                 const void* v, const float* g, const void* beta,
                                 const void* beta_tilde, const float* d, const float* h0, float* o,
                                 float* ht, void* stream) {
  return recurrent_fwd(shape, q, k, v, g, beta, beta_tilde, d, h0, o, ht, stream);
}

const char* comba_status_string(comba_status s) {
  switch (s) {
    case COMBA_OK: return "ok";
    case COMBA_ERR_NULL: return "a required pointer is NULL";
    case COMBA_ERR_SHAPE: return "unsupported or inconsistent shape";
    case COMBA_ERR_DTYPE: return "unknown dtype";
    case COMBA_ERR_ALIGN: return "misaligned pointer (q/k/v/dO and the [.., dk|dv] fp32 tensors need 16 B, workspace 256 B)";
    case COMBA_ERR_WORKSPACE: return "workspace too small";
    case COMBA_ERR_HIP: return "HIP kernel launch failed";
    case COMBA_ERR_SCRATCH:
      return "problem too large for the static scratch of comba_chunk_fwd_noalloc (80 MiB; "
             "use comba_chunk_fwd with a workspace)";
  }
  return "unknown status";
}

}  // extern "C"
