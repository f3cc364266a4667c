// Internal interface between the host API (comba_api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "comba.h"

namespace comba {

// One chunk of at most 64 tokens of one sequence (len == 0: unused slot).
struct ChunkInfo {
  int32_t tok0, len, seq, pad;
};
// Chunk range and token range of one sequence.
struct SeqInfo {
  int32_t chunk0, nchunks, tok0, len;
};

// Optional per-stage timing hook: mark() is called before every kernel stage
// with its name and once after the last stage with name == nullptr.
struct StageHook {
  void (*mark)(void* ctx, hipStream_t stream, const char* name);
  void* ctx;
};

struct LaunchArgs {
  bool bf16;
  // forward: also leave the backward's state (tables, per-chunk operands,
  // chunk states X and D) in the backward-sized workspace;
  // backward: reuse that state instead of recomputing the forward
  bool saved;
  int dk, dv, H, N, Tseq, Ttot, ncmax;
  const int32_t* cu_seqlens;
  // beta_tilde (feedback strength) is never NULL here: it points at beta when
  // the two are tied; dbeta_tilde NULL means tied (dbeta then holds the sum)
  const void *q, *k, *v, *beta, *beta_tilde, *dO;
  const float *g, *d, *h0, *dht;
  float *o, *ht;
  float *dq, *dk_, *dv_, *dg, *dbeta, *dbeta_tilde, *dd, *dh0;
  // workspace views
  ChunkInfo* cmap;
  SeqInfo* smap;
  int* sorder;  // packed sequences in the order the scans take them (longest first)
  float *Mw, *Aw, *Gw;            // per chunk-head: M, A (64 x 64), G (64)
  float *Xw, *Dw, *Yw, *dRw;      // per chunk-head: X (dk x dv), D (64 x dv), Y, dR
  float* ddp;                     // per chunk-head partial dd
  // bf16 path, per chunk-head: M, A as int16 64 x 64 with one power-of-two
  // scale per row of M (Ms) and per column of A (As), in MFMA fragment order
  // (frag_off in the kernels); the backward also keeps Q^T as dk x 64 bf16
  int16_t *Mq, *Aq;
  float *Ms, *As;
  uint16_t* QTp;
  // bf16 path, per chunk-head: X, Y (dk x dv), D, dR (64 x dv) as int16 with one
  // power-of-two scale per (row, 32-column block) in the matching *s array;
  // each 32-column block is stored on its own: [chunk-head][dv/32][rows][32],
  // scales [chunk-head][dv/32][rows]
  int16_t *Xq, *Dq, *Yq, *dRq;
  float *Xs, *Ds, *Ys, *dRs;
  int16_t* Xfq;  // bf16 path: sink for the state after the last chunk (same layout)
  float* Xfs;    //   and its scales
  // segmented scans (bf16, fixed-length rows; segP > 1 enables them): each
  // row is scanned as segP virtual rows; per virtual row and head the final
  // state from a zero start (segF, dk x dv), the transition product (segPhi,
  // dk x dk), the true state entering it (segX0) and its final state (segHT);
  // backward: the state gradient at its start from a zero end (segG), the
  // true one at its end (segY0) and at its start (segDH0)
  int segP;
  float *segF, *segPhi, *segX0, *segHT, *segG, *segY0, *segDH0;
  SeqInfo* segmap;  // packed sequences: the virtual rows' table (k_seg_map)
  hipStream_t stream;
  StageHook hook;
  void stage(const char* name) const {
    if (hook.mark) hook.mark(hook.ctx, stream, name);
  }
};

hipError_t launch_fwd(const LaunchArgs& a);
hipError_t launch_bwd(const LaunchArgs& a);
// The stateless forward's workspace without the segmented scan's buffers.
size_t fwd_workspace_bytes_plain(const comba_shape* shape);

// Token-by-token recurrence (comba_recurrent_fwd): no workspace.
struct RecurrentArgs {
  bool bf16;
  int dk, dv, H, N, Tseq, Ttot;
  const int32_t* cu_seqlens;
  const void *q, *k, *v, *beta, *beta_tilde;  // beta_tilde never NULL (beta when tied)
  const float *g, *d, *h0;
  float *o, *ht;  // ht may equal h0
  hipStream_t stream;
  StageHook hook;
  void stage(const char* name) const {
    if (hook.mark) hook.mark(hook.ctx, stream, name);
  }
};

hipError_t launch_recurrent(const RecurrentArgs& a);

// Layer input prologue (comba_prologue_fwd / comba_prologue_bwd).
struct PrologueArgs {
  bool bf16;
  int dk, dv, H, N, Tseq, Ttot;
  int nruns;  // 64-token runs of the packed token axis (backward)
  int frun;   // tokens per run of the forward (set by its launcher)
  float eps;
  const int32_t* cu_seqlens;
  const void *xq, *xk, *xv;     // pre-activations (in_dtype)
  const float *wq, *wk, *wv;    // taps [H][d][4]
  void *q, *k, *v;              // forward outputs (in_dtype)
  const float *gq, *gk, *gv;    // backward: gradients of q, k, v
  float *dxq, *dxk, *dxv;       // backward outputs
  float *dwq, *dwk, *dwv;
  float *dwpq, *dwpk, *dwpv;    // per-run dw partials (workspace)
  hipStream_t stream;
  StageHook hook;
  void stage(const char* name) const {
    if (hook.mark) hook.mark(hook.ctx, stream, name);
  }
};

hipError_t launch_prologue(const PrologueArgs& a, bool bwd);
// Output gate over n elements (n a multiple of 4); forward when dy is NULL.
hipError_t launch_gate(bool bf16, long n, const float* o, const void* z, void* y, const float* dy,
                       float* dout, float* dz, hipStream_t st);

}  // namespace comba
