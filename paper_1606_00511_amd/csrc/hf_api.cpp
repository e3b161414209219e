// Host side of the C ABI declared in include/hf.h: context, argument
// validation, workspace carve-up, the order of the passes for the gradient,
// the curvature products and CG-Minimize, and the kernel profiler.
//
// Pass order (B = rows, L = weight layers, A_0 = X):
//   gradient (Alg. 1 step 1):
//     forward   Z_l = A_{l-1} W_l^T + b_l,  A_l = phi(Z_l)          (l < L)
//     output    p = softmax(Z_L), f, delta_L = (p - e_y) / B
//     backward  grad W_l = delta_l^T A_{l-1},  grad b_l = sum_rows delta_l,
//               delta_{l-1} = (delta_l W_l) * phi'(A_{l-1})
//   curvature product (Sec. 2.1, after Alg. 1), v = (V_l, c_l):
//     R-forward RZ_l = A_{l-1} V_l^T + RA_{l-1} W_l^T + c_l,
//               RA_l = phi'(A_l) RZ_l   (fused with the forward GEMM)
//     output    Rdelta_L = p * (RZ_L - rowsum(p * RZ_L)) / B
//     Hessian   (Hv)_{W_l} = Rdelta_l^T A_{l-1} + delta_l^T RA_{l-1},
//               (Hv)_{b_l} = sum_rows Rdelta_l,
//               Rdelta_{l-1} = (Rdelta_l W_l + delta_l V_l) phi'(A_{l-1})
//                              + (delta_l W_l) phi''(A_{l-1}) RZ_{l-1}
//     Gauss-Newton (Gv)_{W_l} = Rdelta_l^T A_{l-1}, (Gv)_{b_l} = sum Rdelta_l,
//               Rdelta_{l-1} = (Rdelta_l W_l) phi'(A_{l-1})
//   CG-Minimize (Alg. 1 steps 3-4): the forward pass, p, delta_l and
//     (delta_l W_l) phi''(A_{l-1}) are computed once on the curvature batch and
//     reused by every product inside the solve.
#include "hf.h"
#include "hf_internal.h"

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <new>
#include <string>
#include <vector>

#ifndef HF_BUILD_ID
#define HF_BUILD_ID "unknown"
#endif

using namespace hfk;

// ------------------------------------------------------------------ profiler
namespace hfk {

struct ProfRec {
  std::string name;
  int64_t launches = 0;
  double ms = 0.0, flops = 0.0, bytes = 0.0;
};

struct Profiler {
  std::vector<ProfRec> recs;
  std::map<std::string, int> index;
  struct Pending { hipEvent_t a, b; int rec; int tag; double flops, bytes; };
  std::vector<Pending> pending;
  std::vector<hipEvent_t> pool;
  hipEvent_t open = nullptr, close = nullptr;   // the pair of the next launch
  std::string only;        // time only launches of this name ("" = all)
  int tag = -1;          // CG iteration of the launches being recorded, -1 outside CG
  size_t solve_begin = 0;  // first pending entry of the CG solve in progress

  hipEvent_t get() {
    if (!pool.empty()) {
      hipEvent_t e = pool.back();
      pool.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
  int rec_of(const char* name) {
    auto it = index.find(name);
    if (it != index.end()) return it->second;
    ProfRec r;
    r.name = name;
    recs.push_back(r);
    index[name] = (int)recs.size() - 1;
    return (int)recs.size() - 1;
  }
  // Launches outside the hf_prof_only filter have null events: counted, not
  // timed.
  void collect() {
    for (auto& p : pending) {
      if (!p.a) continue;
      (void)hipEventSynchronize(p.b);
      float ms = 0.0f;
      if (hipEventElapsedTime(&ms, p.a, p.b) == hipSuccess) recs[p.rec].ms += ms;
      pool.push_back(p.a);
      pool.push_back(p.b);
    }
    pending.clear();
  }
  void release(const Pending& p) {
    if (!p.a) return;
    pool.push_back(p.a);
    pool.push_back(p.b);
  }
  // Drop the launches of a CG solve that the device `done` flag turned into
  // no-ops, so that only launches that did their work are counted.
  // last = the last iteration that evaluated a product; stop_on_kappa: the
  // update kernel of that iteration stopped on kappa (negative curvature or a
  // non-finite value) before touching x and r; neg_iter: the iteration of a
  // detection (-1: none), whose update and direction kernels formed g.p and
  // d~ (without one they did no vector work).
  void retract(int last, bool stop_on_kappa, int neg_iter) {
    std::vector<Pending> keep(pending.begin(), pending.begin() + solve_begin);
    keep.reserve(pending.size());
    for (size_t i = solve_begin; i < pending.size(); ++i) {
      Pending& p = pending[i];
      bool drop = false;
      if (p.tag >= 0) {
        const std::string& nm = recs[p.rec].name;
        // at a detection the update and direction kernels form g.p and d~;
        // at a non-finite kappa they do nothing
        if (p.tag > last) drop = true;
        else if (p.tag == last && stop_on_kappa && neg_iter != last)
          drop = nm == "hf_cg_update" || nm == "hf_cg_dir" ||
                 nm == "hf_pcg_update" || nm == "hf_pcg_dir";
      }
      if (drop) {
        recs[p.rec].launches -= 1;
        recs[p.rec].flops -= p.flops;
        recs[p.rec].bytes -= p.bytes;
        release(p);
      } else {
        keep.push_back(p);
      }
    }
    pending.swap(keep);
  }
  // Bi-CG-STAB: launches are tagged with the index of the curvature product
  // they belong to (2j, 2j+1); drop those past the last product evaluated and
  // the candidate writes of iterations without a detection.
  void retract_bicg(int products, int neg_iter) {
    std::vector<Pending> keep(pending.begin(), pending.begin() + solve_begin);
    for (size_t i = solve_begin; i < pending.size(); ++i) {
      Pending& p = pending[i];
      bool drop = false;
      if (p.tag >= 0) {
        if (p.tag >= products) drop = true;
        else if (recs[p.rec].name == "hf_bicg_negw") drop = p.tag / 2 != neg_iter;
      }
      if (drop) {
        recs[p.rec].launches -= 1;
        recs[p.rec].flops -= p.flops;
        recs[p.rec].bytes -= p.bytes;
        release(p);
      } else {
        keep.push_back(p);
      }
    }
    pending.swap(keep);
  }
  ~Profiler() {
    collect();
    for (auto e : pool) (void)hipEventDestroy(e);
  }
};

void prof_begin(const Launch& L, const char* name) {
  (void)name;
  if (!L.prof) return;
  Profiler& P = *L.prof;
  if (!P.only.empty() && P.only != name) {
    P.open = P.close = nullptr;
    return;
  }
  P.open = P.get();
  P.close = P.get();
  if (!P.open || !P.close) {
    if (P.open) P.pool.push_back(P.open);
    if (P.close) P.pool.push_back(P.close);
    P.open = P.close = nullptr;
  }
}

hipEvent_t prof_a(const Launch& L) { return L.prof ? L.prof->open : nullptr; }
hipEvent_t prof_b(const Launch& L) { return L.prof ? L.prof->close : nullptr; }

void prof_end(const Launch& L, const char* name, double flops, double bytes) {
  if (!L.prof) return;
  Profiler& P = *L.prof;
  const int r = P.rec_of(name);
  P.recs[r].launches += 1;
  P.recs[r].flops += flops;
  P.recs[r].bytes += bytes;
  // every launch gets an entry (null events when it is not timed), so that
  // the no-op launches of a stopped solve are retracted for every name
  P.pending.push_back({P.open, P.close, r, P.tag, flops, bytes});
  P.open = P.close = nullptr;
  if (P.tag < 0 && P.pending.size() > (1u << 16)) P.collect();
}

}  // namespace hfk

// ------------------------------------------------------------------- context
struct hf_ctx {
  int L = 0;                   // weight layers
  std::vector<int> d;          // d_0 .. d_L
  std::vector<int> ld;         // padded leading dimensions (multiple of 4)
  int act = 0, prec = 0;
  int64_t Bmax = 0;
  int64_t Bws = 0;             // rows the workspace layout serves (<= Bmax)
  int64_t n = 0;
  std::vector<int64_t> offW, offB;   // 1-based, parameter offsets
  hipStream_t stream = nullptr;

  // workspace carve-up (byte offsets), 1-based per layer where it applies
  std::vector<size_t> oA, oD, oE2, oRZ, oRA, oRD, oWT, oVT;
  // HF_BF16_INPUTS: bf16 GEMM operands.  Row-major copies have leading
  // dimension ldh_l; the transposed (batch-contiguous) ones *T have ldB.
  std::vector<int> ldh;
  int ldB = 0;
  size_t hbeg = 0, hend = 0;   // the bf16 region, zeroed by hf_set_workspace
  size_t hX = 0, hXT = 0;
  std::vector<size_t> hW, hWT, hV, hVT, hA, hAT, hRA, hRAT, hD, hDT, hRD, hRDT;
  size_t oS = 0, oT = 0, oRs = 0;    // Bi-CG-STAB: s, t = B s, r0*
  size_t oPh = 0, oSh = 0;           // preconditioned: M^-1 p, M^-1 s
  size_t oMv = 0;                    // hf_iterate's M^-1
  // outer iteration: gradient, solver step and direction, warm start,
  // trial weights, and device scalars (4 dot products, the fp64 loss)
  size_t oG = 0, oStep = 0, oNd = 0, oX0 = 0, oWt = 0, oScal = 0;
  size_t oZ = 0, oP = 0, oSplit = 0, oBpart = 0, oR = 0, oPv = 0, oQ = 0,
         oRed = 0, oLoss = 0, oState = 0, oErr = 0, need = 0;
  int max_splits = 32;
  bool cached_layout = false;   // the layout holds the transposed weights
  // concatenated columns for the narrow-net weight gradients (NarrowCat):
  // X, A_1 .. A_{L-1} (Ycat) and RA (RAcat), width ldy; Rdelta (RDcat) and
  // delta (Dcat), width ldr.  cat_B / cat_hess: the batch and mode whose
  // cache build filled Ycat (and Dcat), -1 if none.
  bool narrow_cat = false;
  int ldr_cat = 0, ldy_cat = 0;
  int roff[NARROW_MAX_LAYERS + 1] = {}, yoff[NARROW_MAX_LAYERS + 1] = {};
  size_t oYcat = 0, oRDcat = 0, oDcat = 0, oRAcat = 0;
  int cat_B = -1;
  bool cat_hess = false;
  // a CG iteration's request that its product also form the partials of
  // p.q and p.p (fuse.p set for that one product call); fused_blocks: how
  // many partials it wrote, 0 if the product took a route without them
  CgDotFuse fuse = {};
  int fused_blocks = 0;
  size_t split_floats = 0;  // capacity of the split-K scratch (floats)

  char* ws = nullptr;
  size_t ws_bytes = 0;

  std::string err;
  Profiler* prof = nullptr;
  CgState* pinned = nullptr;       // 2 host-pinned copies of the CG state
  void* pinned_bicg = nullptr;     // 2 host-pinned copies of the Bi-CG-STAB state
  hipEvent_t ev[2] = {nullptr, nullptr};
  // lock-step diagnostic (hf_set_trace): operand and result of the first
  // trace_cap curvature products of every solve
  float* trace_buf = nullptr;
  int trace_cap = 0;
  // the label-error flag, when it lives outside the workspace
  int* err_override = nullptr;
  // layout of the no-allocation entry point's device scratch (made on its
  // first call, re-planned for each call's batch)
  hf_ctx* na = nullptr;
  // one CG iteration (product and vector kernels) captured as a graph and
  // replayed per iteration; rebuilt when an argument it captured changes
  struct CgKey {
    const void *W, *X, *g, *step, *nd, *minv;
    const char* ws;
    int64_t b, Bws;
    int mode;
    bool operator==(const CgKey& o) const {
      return W == o.W && X == o.X && g == o.g && step == o.step && nd == o.nd &&
             minv == o.minv && ws == o.ws && b == o.b && Bws == o.Bws && mode == o.mode;
    }
  };
  hipGraphExec_t cg_exec = nullptr;
  CgKey cg_key = {};
  hipStream_t cap_stream = nullptr;
  int* hflag = nullptr;        // host-pinned stop flag the replayed iteration writes
  int* hflag_dev = nullptr;    // its device address
  bool graphs_off = false;     // capture failed once: use the launch-by-launch loop

  float* F(size_t off) const { return reinterpret_cast<float*>(ws + off); }
  double* Dp(size_t off) const { return reinterpret_cast<double*>(ws + off); }
  bf16_t* H(size_t off) const { return reinterpret_cast<bf16_t*>(ws + off); }
  bool bf16() const { return prec == HF_BF16_INPUTS; }
  int* errp() const {
    return err_override ? err_override : reinterpret_cast<int*>(ws + oErr);
  }
  Launch launch() const { return Launch{stream, prof}; }
};

namespace {

int fail(hf_ctx* c, int code, const char* fmt, ...) __attribute__((format(printf, 3, 4)));
int fail(hf_ctx* c, int code, const char* fmt, ...) {
  if (c) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    c->err = buf;
  }
  return code;
}

#define HIP_TRY(ctx, expr)                                                     \
  do {                                                                         \
    hipError_t e_ = (expr);                                                    \
    if (e_ != hipSuccess)                                                      \
      return fail(ctx, HF_EHIP, "%s failed: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

inline size_t up256(size_t x) { return (x + 255) & ~size_t(255); }
inline bool a16(const void* p) { return ((uintptr_t)p & 15u) == 0; }
inline int round4(int x) { return (x + 3) & ~3; }
inline int round64(int x) { return (x + 63) & ~63; }
inline size_t round256(size_t x) { return (x + 255) & ~size_t(255); }

// Carve the workspace for calls of up to B rows (B <= Bmax).  A
// product-only layout holds what a stateless curvature product uses: no
// transposed weights (fp32) and no solver vectors or state.
void plan(hf_ctx* c, int64_t Bplan, bool product_only = false) {
  c->Bws = Bplan;
  c->cached_layout = !product_only;
  c->ldB = round64((int)Bplan);
  const int L = c->L;
  const bool h = c->bf16();
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += up256(bytes);
    return o;
  };
  const size_t B = (size_t)Bplan;
  for (auto* v : {&c->oA, &c->oD, &c->oE2, &c->oRZ, &c->oRA, &c->oRD, &c->oWT,
                  &c->oVT, &c->hW, &c->hWT, &c->hV, &c->hVT, &c->hA, &c->hAT,
                  &c->hRA, &c->hRAT, &c->hD, &c->hDT, &c->hRD, &c->hRDT})
    v->assign(L + 1, 0);
  const size_t f4 = sizeof(float), h2 = sizeof(bf16_t);
  const size_t LB = (size_t)c->ldB;
  // bf16 operands (and the fp32 rows the bf16 epilogues read) have rows up
  // to a multiple of 256: the GEMM tiles read them without bounds checks
  const size_t RB = h ? round256(B) : B;
  auto R256 = [&](int d) { return round256((size_t)d); };
  if (!h && !product_only) {
    for (int l = 1; l <= L; ++l) {
      // W_l and V_l transposed: d_{l-1} rows of ld_l floats
      c->oWT[l] = take((size_t)c->d[l - 1] * c->ld[l] * f4);
      c->oVT[l] = take((size_t)c->d[l - 1] * c->ld[l] * f4);
    }
  } else if (h) {
    c->hbeg = off;
    for (int l = 1; l <= L; ++l) {
      // bf16 W_l, V_l (row-major, forward) and transposed (backward)
      c->hW[l] = take(R256(c->d[l]) * c->ldh[l - 1] * h2);
      c->hWT[l] = take(R256(c->d[l - 1]) * c->ldh[l] * h2);
      c->hV[l] = take(R256(c->d[l]) * c->ldh[l - 1] * h2);
      c->hVT[l] = take(R256(c->d[l - 1]) * c->ldh[l] * h2);
    }
    c->hX = take(RB * c->ldh[0] * h2);
    c->hXT = take(R256(c->d[0]) * LB * h2);
    for (int l = 1; l <= L; ++l) {
      const size_t szh = RB * c->ldh[l] * h2, szt = R256(c->d[l]) * LB * h2;
      if (l < L) {
        c->hA[l] = take(szh);
        c->hAT[l] = take(szt);
        c->hRA[l] = take(szh);
        c->hRAT[l] = take(szt);
      }
      c->hD[l] = take(szh);
      c->hDT[l] = take(szt);
      c->hRD[l] = take(szh);
      c->hRDT[l] = take(szt);
    }
    c->hend = off;
  }
  for (int l = 1; l <= L; ++l) {
    const size_t sz = RB * c->ld[l] * f4;
    if (!h) {
      if (l < L) {
        c->oA[l] = take(sz);
        c->oE2[l] = take(sz);
        c->oRA[l] = take(sz);
      }
      c->oD[l] = take(sz);
      c->oRZ[l] = take(sz);
      c->oRD[l] = take(sz);
    } else {
      if (l < L) c->oE2[l] = take(sz);
      else {
        c->oD[l] = take(sz);     // fp32 softmax outputs, converted to bf16
        c->oRD[l] = take(sz);
      }
      c->oRZ[l] = take(sz);
    }
  }
  c->oZ = take(RB * c->ld[L] * f4);
  c->oP = take(RB * c->ld[L] * f4);
  // narrow nets: the concatenated columns of their weight-gradient GEMM
  c->narrow_cat = false;
  c->cat_B = -1;
  if (!h && !product_only && narrow_eligible(L, c->d.data(), nullptr, nullptr)) {
    c->narrow_cat = true;
    int r = 0, y = 0;
    for (int l = 1; l <= L; ++l) { c->roff[l] = r; r += round4(c->d[l]); }
    for (int l = 0; l < L; ++l) { c->yoff[l] = y; y += round4(c->d[l]); }
    c->ldr_cat = r;
    c->ldy_cat = y;
    c->oYcat = take(B * (size_t)y * f4);
    c->oRAcat = take(B * (size_t)y * f4);
    c->oRDcat = take(B * (size_t)r * f4);
    c->oDcat = take(B * (size_t)r * f4);
  }
  // Split-K scratch.  A weight gradient (d_l x d_{l-1}, K up to 2 B rows
  // over two segments) takes at most the splits that keep every split within
  // 2,048 rows at that K (bf16: fewer), or, if the tile rule asked for
  // more, fewer than 1,024 tiles of 128 x 128 worth of partials (bf16: 512
  // tiles of 256 x 256).  A batch-row GEMM splits only while its grid holds
  // fewer than 512 tiles, so it too stays below 1,024 tiles' worth (and below
  // max_splits x B x the widest layer).  With this much scratch no split is
  // cut short.  (The bf16 batch-row GEMMs do not split.)
  const size_t TILES_1024 = (size_t)1024 * 128 * 128 * (h ? 2 : 1);
  int dmax = 0;
  size_t wg = 0;
  for (int l = 1; l <= L; ++l) {
    const size_t mn = (size_t)c->d[l] * c->d[l - 1];
    int s1 = 1;
    while (s1 < c->max_splits && (2 * B + s1 - 1) / s1 > 2048) s1 *= 2;
    wg = std::max(wg, std::min((size_t)c->max_splits * mn,
                               std::max((size_t)s1 * mn, TILES_1024)));
    dmax = std::max(dmax, c->d[l]);
  }
  const size_t rows = h ? 0 : std::min(TILES_1024, (size_t)c->max_splits * B * (size_t)dmax);
  c->split_floats = std::max(wg, rows);
  // the narrow nets' concatenated weight-gradient GEMM (at most max_splits
  // partials of ldr x ldy)
  if (c->narrow_cat)
    c->split_floats = std::max(c->split_floats,
                               (size_t)c->max_splits * c->ldr_cat * c->ldy_cat);
  c->oSplit = take(c->split_floats * f4);

  c->oBpart = take((size_t)c->max_splits * std::max(dmax, c->narrow_cat ? c->ldr_cat : 0) *
                   sizeof(double));
  c->oLoss = take(((B + 3) / 4) * sizeof(double));
  c->oErr = take(sizeof(int));
  if (product_only) {
    c->oR = c->oPv = c->oQ = c->oS = c->oT = c->oRs = c->oPh = c->oSh = c->oMv =
        c->oG = c->oStep = c->oNd = c->oX0 = c->oWt = c->oScal = c->oRed =
            c->oState = 0;
    c->need = off;
    return;
  }
  const size_t nv = ((size_t)c->n + 63) & ~size_t(63);
  c->oR = take(nv * f4);
  c->oPv = take(nv * f4);
  c->oQ = take(nv * f4);
  c->oS = take(nv * f4);
  c->oT = take(nv * f4);
  c->oRs = take(nv * f4);
  c->oPh = take(nv * f4);
  c->oSh = take(nv * f4);
  c->oMv = take(nv * f4);
  c->oG = take(nv * f4);
  c->oStep = take(nv * f4);
  c->oNd = take(nv * f4);
  c->oX0 = take(nv * f4);
  c->oWt = take(nv * f4);
  c->oScal = take(8 * sizeof(double));
  c->oRed = take((size_t)cg_part_doubles() * sizeof(double));
  c->oState = take(sizeof(CgState) > sizeof(BicgState) ? sizeof(CgState)
                                                        : sizeof(BicgState));
  c->need = off;
}

bool valid_act(int a) { return a == HF_SIGMOID || a == HF_TANH || a == HF_RELU; }

int check_ready(hf_ctx* c) {
  if (!c) return HF_EINVAL;
  if (!c->ws) return fail(c, HF_EWORKSPACE, "no workspace set (hf_set_workspace)");
  return HF_OK;
}

int check_ptr(hf_ctx* c, const void* p, const char* what) {
  if (!p) return fail(c, HF_EINVAL, "%s is NULL", what);
  if (!a16(p)) return fail(c, HF_EINVAL, "%s is not 16-byte aligned", what);
  return HF_OK;
}

int check_batch(hf_ctx* c, int64_t B) {
  if (B < 1 || B > c->Bmax)
    return fail(c, HF_EINVAL, "batch %lld outside [1, %lld]", (long long)B,
                (long long)c->Bmax);
  if (B > c->Bws)
    return fail(c, HF_EWORKSPACE, "batch %lld above the %lld rows the workspace serves",
                (long long)B, (long long)c->Bws);
  return HF_OK;
}

// Bytes of workspace for calls of up to B rows (product_only: the layout of
// a stateless curvature product alone).
size_t plan_bytes(const hf_ctx* c, int64_t B, bool product_only = false) {
  hf_ctx t;
  t.L = c->L;
  t.d = c->d;
  t.ld = c->ld;
  t.ldh = c->ldh;
  t.act = c->act;
  t.prec = c->prec;
  t.Bmax = c->Bmax;
  t.n = c->n;
  t.max_splits = c->max_splits;
  plan(&t, B, product_only);
  return t.need;
}

// Operand and result of the k-th curvature product of a solve into the
// trace buffer (hf_set_trace), unless the solve has stopped (skip).
void trace_product(hf_ctx* c, int k, const float* v, const float* out,
                   const int* skip) {
  if (!c->trace_buf || k >= c->trace_cap) return;
  const size_t n = (size_t)c->n;
  keep_iterate(c->launch(), c->trace_buf + (2 * (size_t)k) * n, v, (long long)n, skip);
  keep_iterate(c->launch(), c->trace_buf + (2 * (size_t)k + 1) * n, out, (long long)n,
               skip);
}

// split-K factor for a weight-gradient GEMM with the given tile count and
// reduction length.  First, no split accumulates more than 2,048 rows in
// fp32 (the weight gradients are batch means with heavy cancellation, and the
// splits are combined in fixed order in the reduce kernel); with bf16
// operands 8,192 rows, since their rounding (2^-9 relative per operand)
// outweighs that of fp32 accumulation over 8,192 terms many times over.
// Then, enough workgroups to cover the 256 compute units twice (fp32: 4
// workgroups fit a CU), or once (bf16: its 256 x 256 tiles take one CU each,
// so that each further round of workgroups adds an epilogue and partials
// without adding MFMA throughput), while every split keeps at least 64 rows
// (4 K blocks: enough to fill the load pipeline; a few workgroups with long K
// chains would leave most of the chip idle).
int choose_splits(const hf_ctx* c, int M, int N, int Ktot) {
  const bool h = c->bf16();
  const int ts = h ? 256 : gemm_tile(M, N, Ktot);
  const int tiles = ((M + ts - 1) / ts) * ((N + ts - 1) / ts);
  const int chain = h ? 8192 : 2048, cover = h ? 256 : 512;
  int s = 1;
  while (s < c->max_splits && (Ktot + s - 1) / s > chain) s *= 2;
  while (s < c->max_splits && tiles * s < cover && Ktot / (2 * s) >= 64) s *= 2;
  // the scratch is sized so that this never applies; it keeps the partials
  // in bounds regardless
  while (s > 1 && (size_t)s * M * N > c->split_floats) s /= 2;
  return s;
}

GemmShape shape(int M, int N, int K, const float* x0, const float* x1,
                const float* y0, const float* y1, int ldx, int ldy, int nseg,
                const int* skip) {
  GemmShape s;
  s.M = M; s.N = N; s.K = K;
  s.X[0] = x0; s.X[1] = x1;
  s.Y[0] = y0; s.Y[1] = y1;
  s.ldx = ldx; s.ldy = ldy;
  s.nseg = nseg;
  s.splits = 1;
  s.skip = skip;
  return s;
}

EpiArgs epi(const hf_ctx* c, int hidden) {
  EpiArgs e;
  std::memset(&e, 0, sizeof e);
  e.act = c->act;
  e.hidden = hidden;
  e.split_buf = c->F(c->oSplit);
  e.split_cap = (long long)c->split_floats;
  return e;
}

// Weight-gradient GEMM into the parameter layout: out_W (d_l x d_{l-1}) =
// sum_seg Xs^T Ys over the rows, and out_b = column sums of x0 (the first
// segment's X operand), both from the same kernel.
void wgrad(hf_ctx* c, int l, int B, const float* x0, const float* y0,
           const float* x1, const float* y1, int ldy, float* out,
           const int* skip, bool sq = false) {
  const Launch Lc = c->launch();
  const int M = c->d[l], N = c->d[l - 1];
  const int nseg = x1 ? 2 : 1;
  GemmShape s = shape(M, N, B, x0, x1, y0, y1, c->ld[l], ldy, nseg, skip);
  s.splits = choose_splits(c, M, N, B * nseg);
  EpiArgs e = epi(c, 0);
  e.ldo = N;
  if (s.splits > 1) {
    e.out0 = c->F(c->oSplit);
    e.split_stride = (long long)M * N;
    e.bias_part = c->Dp(c->oBpart);
    (sq ? gemm_wgrad_sq : gemm_wgrad)(Lc, s, e);
    splitk_reduce(Lc, c->F(c->oSplit), c->Dp(c->oBpart), s.splits, M, N,
                  out + c->offW[l], N, out + c->offB[l], skip);
  } else {
    e.out0 = out + c->offW[l];
    e.bias_out = out + c->offB[l];
    (sq ? gemm_wgrad_sq : gemm_wgrad)(Lc, s, e);
  }
}

// Weight blocks of a parameter-layout vector, transposed to [d_{l-1}][ld_l]
// (the row-contiguous right operand of the forward GEMMs).
void transpose_weights(hf_ctx* c, const float* v, const std::vector<size_t>& dst,
                       const int* skip) {
  TransposeBatch b;
  static_assert(TransposeBatch::MAX >= HF_MAX_LAYERS, "one block per layer");
  b.n = c->L;
  for (int l = 1; l <= c->L; ++l) {
    const int i = l - 1;
    b.in[i] = v + c->offW[l];
    b.R[i] = c->d[l];
    b.C[i] = c->d[l - 1];
    b.ldi[i] = c->d[l - 1];
    b.out[i] = c->F(dst[l]);
    b.ldo[i] = c->ld[l];
  }
  transpose_batch(c->launch(), b, skip);
}

// Forward pass (activations only) on B rows of X; logits into Z, then the
// softmax / cross-entropy kernel (labels optional).
void forward_plain(hf_ctx* c, const float* W, const float* X, int B,
                   const int32_t* y, bool want_delta) {
  const Launch Lc = c->launch();
  c->cat_B = -1;   // the concatenated copy no longer matches the cache
  transpose_weights(c, W, c->oWT, nullptr);
  for (int l = 1; l <= c->L; ++l) {
    const float* Ain = (l == 1) ? X : c->F(c->oA[l - 1]);
    const int ldin = (l == 1) ? c->d[0] : c->ld[l - 1];
    GemmShape s = shape(B, c->d[l], c->d[l - 1], Ain, nullptr, c->F(c->oWT[l]),
                        nullptr, ldin, c->ld[l], 1, nullptr);
    EpiArgs e = epi(c, l < c->L);
    e.bias = W + c->offB[l];
    e.out0 = (l < c->L) ? c->F(c->oA[l]) : c->F(c->oZ);
    e.ldo = c->ld[l];
    gemm_fwd(Lc, s, e);
  }
  softmax_xent(Lc, c->F(c->oZ), y, B, c->d[c->L], c->ld[c->L], c->F(c->oP),
               want_delta ? c->F(c->oD[c->L]) : nullptr, c->Dp(c->oLoss),
               c->errp());
}

// Backward data pass delta_{l-1} = (delta_l W_l) phi'(A_{l-1}); optionally
// caches (delta_l W_l) phi''(A_{l-1}) for the Hessian product.
void backward_data(hf_ctx* c, const float* W, int l, int B, bool cache_e2) {
  GemmShape s = shape(B, c->d[l - 1], c->d[l], c->F(c->oD[l]), nullptr,
                      W + c->offW[l], nullptr, c->ld[l], c->d[l - 1], 1, nullptr);
  EpiArgs e = epi(c, 1);
  e.out0 = c->F(c->oD[l - 1]);
  e.out2 = cache_e2 ? c->F(c->oE2[l - 1]) : nullptr;
  e.ldo = c->ld[l - 1];
  e.aux0 = c->F(c->oA[l - 1]);
  e.lda = c->ld[l - 1];
  gemm_bwd(c->launch(), s, e);
}

// Every layer's weight gradient of a narrow net from one GEMM over the
// concatenated columns: x0 (width ldr) against Ycat (width ldy), plus x1
// against y1 when given (the Hessian's second term), over B rows; then the
// scatter of the diagonal blocks into out (parameter layout).  Returns the
// scatter's count of CG dot partials (dot: a CG iteration's request).
int cat_wgrad(hf_ctx* c, int B, const float* x0, const float* x1, const float* y1,
              float* out, const int* skip, const CgDotFuse* dot) {
  const int L = c->L;
  const int M = c->ldr_cat, N = c->ldy_cat;
  GemmShape s = shape(M, N, B, x0, x1, c->F(c->oYcat), y1, M, N, x1 ? 2 : 1, skip);
  // always through the partials, so that the scatter has them
  s.splits = std::max(2, choose_splits(c, M, N, B * s.nseg));
  EpiArgs e = epi(c, 0);
  e.out0 = c->F(c->oSplit);
  e.ldo = N;
  e.split_stride = (long long)M * N;
  e.bias_part = c->Dp(c->oBpart);
  gemm_wgrad(c->launch(), s, e);
  NarrowCat nc;
  std::memset(&nc, 0, sizeof nc);
  nc.L = L;
  nc.M = M;
  nc.N = N;
  for (int l = 0; l <= L; ++l) {
    nc.d[l] = c->d[l];
    nc.roff[l] = c->roff[l];
    nc.yoff[l] = c->yoff[l];
    if (l >= 1) {
      nc.offW[l] = c->offW[l];
      nc.offB[l] = c->offB[l];
    }
  }
  nc.offW[L + 1] = c->n;
  nc.n = c->n;
  return narrow_scatter(c->launch(), c->F(c->oSplit), c->Dp(c->oBpart), s.splits, nc, out,
                        skip, dot);
}

// One curvature product out = A v on B rows of X with the forward cache
// (A_l, p, delta_l, E2_l and the transposed weights) already computed;
// skip = device flag or null.
// The narrow-net form of product_cached: one launch up to the weight
// gradients, where its grid of 16-row workgroups beats the GEMM path (the
// small-output regime of the first layer's GEMM).
bool product_narrow(hf_ctx* c, const float* W, const float* X, int B,
                    const float* v, int mode, float* out, const int* skip) {
  const int L = c->L;
  if (!narrow_eligible(L, c->d.data(), X, v) || gemm_tile(B, c->d[1], c->d[0]) != 64)
    return false;
  const bool hess = mode == HF_HESSIAN;
  NarrowArgs a;
  std::memset(&a, 0, sizeof a);
  a.L = L;
  a.B = B;
  a.act = c->act;
  a.hess = hess ? 1 : 0;
  for (int l = 0; l <= L; ++l) {
    a.d[l] = c->d[l];
    a.ld[l] = l == 0 ? c->d[0] : c->ld[l];
    a.offW[l] = l == 0 ? 0 : (long long)c->offW[l];
    a.offB[l] = l == 0 ? 0 : (long long)c->offB[l];
    if (l >= 1) a.RD[l] = c->F(c->oRD[l]);
    if (l >= 1 && l < L) {
      a.A[l] = c->F(c->oA[l]);
      a.RA[l] = c->F(c->oRA[l]);
      a.E2[l] = hess ? c->F(c->oE2[l]) : nullptr;
    }
    if (l >= 2) a.D[l] = hess ? c->F(c->oD[l]) : nullptr;
  }
  a.X = X;
  a.W = W;
  a.RZ1 = c->F(c->oRZ[1]);
  a.v = v;
  a.P = c->F(c->oP);
  a.invB = 1.0f / (float)B;
  a.skip = skip;
  const bool cat = c->cat_B == B && (!hess || c->cat_hess);
  if (cat) {
    // every layer's Rdelta (and RA) into the concatenated columns, then one
    // weight-gradient GEMM for all layers and the scatter of its diagonal
    // blocks
    a.ldRD = c->ldr_cat;
    a.ldRA = c->ldy_cat;
    for (int l = 1; l <= L; ++l) {
      a.RD[l] = c->F(c->oRDcat) + c->roff[l];
      if (l < L) a.RA[l] = c->F(c->oRAcat) + c->yoff[l];
    }
    narrow_product(c->launch(), a);
    c->fused_blocks = cat_wgrad(c, B, c->F(c->oRDcat), hess ? c->F(c->oDcat) : nullptr,
                                hess ? c->F(c->oRAcat) : nullptr, out, skip,
                                c->fuse.p == v ? &c->fuse : nullptr);
    return true;
  }
  narrow_product(c->launch(), a);
  for (int l = L; l >= 1; --l) {
    const float* Ain = (l == 1) ? X : c->F(c->oA[l - 1]);
    const int ldin = (l == 1) ? c->d[0] : c->ld[l - 1];
    if (hess && l > 1)
      wgrad(c, l, B, c->F(c->oRD[l]), Ain, c->F(c->oD[l]), c->F(c->oRA[l - 1]),
            ldin, out, skip);
    else
      wgrad(c, l, B, c->F(c->oRD[l]), Ain, nullptr, nullptr, ldin, out, skip);
  }
  return true;
}

void product_cached(hf_ctx* c, const float* W, const float* X, int B,
                    const float* v, int mode, float* out, const int* skip) {
  const Launch Lc = c->launch();
  const int L = c->L;
  if (product_narrow(c, W, X, B, v, mode, out, skip)) return;
  transpose_weights(c, v, c->oVT, skip);
  for (int l = 1; l <= L; ++l) {
    GemmShape s;
    if (l == 1) {
      s = shape(B, c->d[1], c->d[0], X, nullptr, c->F(c->oVT[1]), nullptr,
                c->d[0], c->ld[1], 1, skip);
    } else {
      s = shape(B, c->d[l], c->d[l - 1], c->F(c->oRA[l - 1]), c->F(c->oA[l - 1]),
                c->F(c->oWT[l]), c->F(c->oVT[l]), c->ld[l - 1], c->ld[l], 2, skip);
    }
    EpiArgs e = epi(c, l < L);
    e.rbias = v + c->offB[l];
    // RZ_l is read by the softmax R-op (l = L) and by the Hessian's
    // R-backward; the Gauss-Newton product needs only RA_l of a hidden layer
    e.out1 = (l == L || mode == HF_HESSIAN) ? c->F(c->oRZ[l]) : nullptr;
    e.out2 = (l < L) ? c->F(c->oRA[l]) : nullptr;
    e.ldo = c->ld[l];
    e.aux0 = (l < L) ? c->F(c->oA[l]) : nullptr;
    e.lda = c->ld[l];
    gemm_rfwd(Lc, s, e);
  }
  softmax_rop(Lc, c->F(c->oP), c->F(c->oRZ[L]), B, c->d[L], c->ld[L],
              c->F(c->oRD[L]), skip);
  for (int l = L; l >= 1; --l) {
    const float* Ain = (l == 1) ? X : c->F(c->oA[l - 1]);
    const int ldin = (l == 1) ? c->d[0] : c->ld[l - 1];
    if (mode == HF_HESSIAN && l > 1) {
      wgrad(c, l, B, c->F(c->oRD[l]), Ain, c->F(c->oD[l]), c->F(c->oRA[l - 1]),
            ldin, out, skip);
    } else {
      wgrad(c, l, B, c->F(c->oRD[l]), Ain, nullptr, nullptr, ldin, out, skip);
    }
    if (l == 1) break;
    EpiArgs e = epi(c, 1);
    e.out1 = c->F(c->oRD[l - 1]);
    e.ldo = c->ld[l - 1];
    e.aux0 = c->F(c->oA[l - 1]);
    e.lda = c->ld[l - 1];
    if (mode == HF_HESSIAN) {
      GemmShape s = shape(B, c->d[l - 1], c->d[l], c->F(c->oRD[l]), c->F(c->oD[l]),
                          W + c->offW[l], v + c->offW[l], c->ld[l], c->d[l - 1],
                          2, skip);
      e.aux1 = c->F(c->oRZ[l - 1]);
      e.aux2 = c->F(c->oE2[l - 1]);
      gemm_rbwd(Lc, s, e);
    } else {
      GemmShape s = shape(B, c->d[l - 1], c->d[l], c->F(c->oRD[l]), nullptr,
                          W + c->offW[l], nullptr, c->ld[l], c->d[l - 1], 1, skip);
      gemm_gnbwd(Lc, s, e);
    }
  }
}

// ------------------------------------------------- bf16-input passes
// The same pass order as above with every GEMM operand a bf16 copy.  The
// producing epilogues write each bf16 activation or delta twice: row-major
// (the next forward or backward GEMM's operand) and transposed (the weight
// gradient's batch-contiguous operand); RA, which only the Hessian's weight
// gradient reads transposed, is stored once in a Gauss-Newton product.
// Softmax, RZ, the phi'' cache and all reductions stay fp32.

EpiH epih(const hf_ctx* c, int hidden) {
  EpiH e;
  std::memset(&e, 0, sizeof e);
  e.act = c->act;
  e.hidden = hidden;
  e.ldt = c->ldB;
  return e;
}

GemmShapeH shapeh(int M, int N, int K, const bf16_t* x0, const bf16_t* x1,
                  const bf16_t* y0, const bf16_t* y1, int ldx, int ldy,
                  int nseg, const int* skip) {
  GemmShapeH s;
  s.M = M; s.N = N; s.K = K;
  s.X[0] = x0; s.X[1] = x1;
  s.Y[0] = y0; s.Y[1] = y1;
  s.ldx = ldx; s.ldy = ldy;
  s.nseg = nseg;
  s.splits = 1;
  s.skip = skip;
  return s;
}

// bf16 copies of the weight blocks of a parameter-layout vector: W_l
// row-major [d_l][ldh_{l-1}] and transposed [d_{l-1}][ldh_l]
// (tr null: no transposed copy; a Gauss-Newton product's direction V is
// read only row-major, by the R-forward)
void weights_h(hf_ctx* c, const float* v, const std::vector<size_t>& row,
               const std::vector<size_t>* tr, const int* skip) {
  for (int l = 1; l <= c->L; ++l)
    cvt_bf16(c->launch(), v + c->offW[l], c->d[l], c->d[l - 1], c->d[l - 1],
             c->H(row[l]), c->ldh[l - 1], tr ? c->H((*tr)[l]) : nullptr, c->ldh[l],
             c->ldh[l], skip);
}

// bf16 copies of the input rows: X [B][ldh_0] and X^T [d_0][ldB]
void input_h(hf_ctx* c, const float* X, int B) {
  cvt_bf16(c->launch(), X, B, c->d[0], c->d[0], c->H(c->hX), c->ldh[0],
           c->H(c->hXT), c->ldB, round64(B), nullptr);
}

// Rdelta_L of a bf16-operand product: the softmax R-op writes its bf16
// row-major copy, then the transposed copy is made from that (the fp32
// Rdelta_L is not needed)
void rop_h(hf_ctx* c, int B, const int* skip) {
  const int L = c->L;
  softmax_rop_h(c->launch(), c->F(c->oP), c->F(c->oRZ[L]), B, c->d[L], c->ld[L],
                c->H(c->hRD[L]), c->ldh[L], skip);
  transpose_bf16(c->launch(), c->H(c->hRD[L]), B, c->d[L], c->ldh[L], c->H(c->hRDT[L]),
                 c->ldB, round64(B), skip);
}

// an fp32 output-layer delta (B x d_L, ld_L) to its two bf16 copies
void delta_h(hf_ctx* c, const float* D, int B, size_t row, size_t tr,
             const int* skip) {
  const int L = c->L;
  cvt_bf16(c->launch(), D, B, c->d[L], c->ld[L], c->H(row), c->ldh[L],
           c->H(tr), c->ldB, round64(B), skip);
}

const bf16_t* act_h(const hf_ctx* c, int l) {       // A_l, row-major
  return c->H(l == 0 ? c->hX : c->hA[l]);
}
const bf16_t* act_ht(const hf_ctx* c, int l) {      // A_l, transposed
  return c->H(l == 0 ? c->hXT : c->hAT[l]);
}

void wgrad_h(hf_ctx* c, int l, int B, const bf16_t* x0, const bf16_t* y0,
             const bf16_t* x1, const bf16_t* y1, float* out, const int* skip) {
  const Launch Lc = c->launch();
  const int M = c->d[l], N = c->d[l - 1];
  const int nseg = x1 ? 2 : 1;
  GemmShapeH s = shapeh(M, N, B, x0, x1, y0, y1, c->ldB, c->ldB, nseg, skip);
  s.splits = choose_splits(c, M, N, B * nseg);
  EpiH e = epih(c, 0);
  e.ldf = N;
  if (s.splits > 1) {
    e.f0 = c->F(c->oSplit);
    e.split_stride = (long long)M * N;
    e.bias_part = c->Dp(c->oBpart);
    hgemm_wgrad(Lc, s, e);
    splitk_reduce(Lc, c->F(c->oSplit), c->Dp(c->oBpart), s.splits, M, N,
                  out + c->offW[l], N, out + c->offB[l], skip);
  } else {
    e.f0 = out + c->offW[l];
    e.bias_out = out + c->offB[l];
    hgemm_wgrad(Lc, s, e);
  }
}

void forward_plain_h(hf_ctx* c, const float* W, const float* X, int B,
                     const int32_t* y, bool want_delta) {
  const Launch Lc = c->launch();
  const int L = c->L;
  input_h(c, X, B);
  weights_h(c, W, c->hW, &c->hWT, nullptr);
  for (int l = 1; l <= L; ++l) {
    GemmShapeH s = shapeh(B, c->d[l], c->d[l - 1], act_h(c, l - 1), nullptr,
                          c->H(c->hW[l]), nullptr, c->ldh[l - 1], c->ldh[l - 1],
                          1, nullptr);
    EpiH e = epih(c, l < L);
    e.bias = W + c->offB[l];
    if (l < L) {
      e.h0 = c->H(c->hA[l]);
      e.t0 = c->H(c->hAT[l]);
      e.ldo = c->ldh[l];
    } else {
      e.f0 = c->F(c->oZ);
      e.ldf = c->ld[L];
    }
    hgemm_fwd(Lc, s, e);
  }
  softmax_xent(Lc, c->F(c->oZ), y, B, c->d[L], c->ld[L], c->F(c->oP),
               want_delta ? c->F(c->oD[L]) : nullptr, c->Dp(c->oLoss),
               c->errp());
  if (want_delta) delta_h(c, c->F(c->oD[L]), B, c->hD[L], c->hDT[L], nullptr);
}

void backward_data_h(hf_ctx* c, int l, int B, bool cache_e2) {
  GemmShapeH s = shapeh(B, c->d[l - 1], c->d[l], c->H(c->hD[l]), nullptr,
                        c->H(c->hWT[l]), nullptr, c->ldh[l], c->ldh[l], 1,
                        nullptr);
  EpiH e = epih(c, 1);
  e.h0 = c->H(c->hD[l - 1]);
  e.t0 = c->H(c->hDT[l - 1]);
  e.ldo = c->ldh[l - 1];
  e.a0 = c->H(c->hA[l - 1]);
  e.f2 = cache_e2 ? c->F(c->oE2[l - 1]) : nullptr;
  e.ldf = c->ld[l - 1];
  hgemm_bwd(c->launch(), s, e);
}

// weight gradients of a curvature product at layer l (both modes) and, for
// l > 1, the backward step to Rdelta_{l-1} (and delta_{l-1} when stateless)
void rbackward_h(hf_ctx* c, int l, int B, int mode, bool stateless,
                 float* out, const int* skip) {
  const bool hess = mode == HF_HESSIAN;
  if (hess && l > 1)
    wgrad_h(c, l, B, c->H(c->hRDT[l]), act_ht(c, l - 1), c->H(c->hDT[l]),
            c->H(c->hRAT[l - 1]), out, skip);
  else
    wgrad_h(c, l, B, c->H(c->hRDT[l]), act_ht(c, l - 1), nullptr, nullptr,
            out, skip);
  if (l == 1) return;
  EpiH e = epih(c, 1);
  e.h1 = c->H(c->hRD[l - 1]);
  e.t1 = c->H(c->hRDT[l - 1]);
  e.ldo = c->ldh[l - 1];
  e.a0 = c->H(c->hA[l - 1]);
  e.ldf = c->ld[l - 1];
  const int ld = c->ldh[l];
  if (hess && stateless) {
    // (E, RE) = (delta W, Rdelta W + delta V) in one pass
    GemmShapeH s = shapeh(B, c->d[l - 1], c->d[l], c->H(c->hD[l]),
                          c->H(c->hRD[l]), c->H(c->hWT[l]), c->H(c->hVT[l]),
                          ld, ld, 1, skip);
    e.h0 = c->H(c->hD[l - 1]);
    e.t0 = c->H(c->hDT[l - 1]);
    e.a1 = c->F(c->oRZ[l - 1]);
    hgemm_bwd_rbwd(c->launch(), s, e);
  } else if (hess) {
    GemmShapeH s = shapeh(B, c->d[l - 1], c->d[l], c->H(c->hRD[l]),
                          c->H(c->hD[l]), c->H(c->hWT[l]), c->H(c->hVT[l]), ld,
                          ld, 2, skip);
    e.a1 = c->F(c->oRZ[l - 1]);
    e.a2 = c->F(c->oE2[l - 1]);
    hgemm_rbwd(c->launch(), s, e);
  } else {
    GemmShapeH s = shapeh(B, c->d[l - 1], c->d[l], c->H(c->hRD[l]), nullptr,
                          c->H(c->hWT[l]), nullptr, ld, ld, 1, skip);
    hgemm_gnbwd(c->launch(), s, e);
  }
}

void product_cached_h(hf_ctx* c, int B, const float* v, int mode, float* out,
                      const int* skip) {
  const Launch Lc = c->launch();
  const int L = c->L;
  weights_h(c, v, c->hV, mode == HF_HESSIAN ? &c->hVT : nullptr, skip);
  for (int l = 1; l <= L; ++l) {
    GemmShapeH s;
    if (l == 1)
      s = shapeh(B, c->d[1], c->d[0], c->H(c->hX), nullptr, c->H(c->hV[1]),
                 nullptr, c->ldh[0], c->ldh[0], 1, skip);
    else
      s = shapeh(B, c->d[l], c->d[l - 1], c->H(c->hRA[l - 1]),
                 c->H(c->hA[l - 1]), c->H(c->hW[l]), c->H(c->hV[l]),
                 c->ldh[l - 1], c->ldh[l - 1], 2, skip);
    EpiH e = epih(c, l < L);
    e.rbias = v + c->offB[l];
    // RZ_l is read by the softmax R-op (l = L) and by the Hessian's
    // R-backward, the transposed RA_l only by the Hessian's weight gradient:
    // the Gauss-Newton product stores RA_l of a hidden layer row-major only
    const bool hess = mode == HF_HESSIAN;
    e.f1 = (l == L || hess) ? c->F(c->oRZ[l]) : nullptr;
    e.ldf = c->ld[l];
    if (l < L) {
      e.h2 = c->H(c->hRA[l]);
      e.t2 = hess ? c->H(c->hRAT[l]) : nullptr;
      e.a0 = c->H(c->hA[l]);
      e.ldo = c->ldh[l];
    }
    hgemm_rfwd(Lc, s, e);
  }
  rop_h(c, B, skip);
  for (int l = L; l >= 1; --l) rbackward_h(c, l, B, mode, false, out, skip);
}

// stateless curvature product: forward fused with R-forward, then the
// R-backward (Hv) or Gauss-Newton backward (Gv)
void hvp_h(hf_ctx* c, const float* W, const float* X, const int32_t* y, int B,
           const float* v, int mode, float* out) {
  const Launch Lc = c->launch();
  const int L = c->L;
  const bool hess = mode == HF_HESSIAN;
  input_h(c, X, B);
  weights_h(c, W, c->hW, &c->hWT, nullptr);
  weights_h(c, v, c->hV, hess ? &c->hVT : nullptr, nullptr);
  for (int l = 1; l <= L; ++l) {
    const int ldk = c->ldh[l - 1];
    GemmShapeH s = shapeh(B, c->d[l], c->d[l - 1], act_h(c, l - 1),
                          l == 1 ? nullptr : c->H(c->hRA[l - 1]),
                          c->H(c->hW[l]), c->H(c->hV[l]), ldk, ldk, 1, nullptr);
    EpiH e = epih(c, l < L);
    e.bias = W + c->offB[l];
    e.rbias = v + c->offB[l];
    // as in the cached product: RZ_l and the transposed RA_l of a hidden
    // layer only for the Hessian
    e.f1 = (l == L || hess) ? c->F(c->oRZ[l]) : nullptr;
    e.ldf = c->ld[l];
    if (l < L) {
      e.h0 = c->H(c->hA[l]);
      e.t0 = c->H(c->hAT[l]);
      e.h2 = c->H(c->hRA[l]);
      e.t2 = hess ? c->H(c->hRAT[l]) : nullptr;
      e.ldo = c->ldh[l];
    } else {
      e.f0 = c->F(c->oZ);
    }
    hgemm_fwd_rfwd(Lc, s, e);
  }
  softmax_xent(Lc, c->F(c->oZ), hess ? y : nullptr, B, c->d[L], c->ld[L],
               c->F(c->oP), hess ? c->F(c->oD[L]) : nullptr, c->Dp(c->oLoss),
               c->errp());
  if (hess) delta_h(c, c->F(c->oD[L]), B, c->hD[L], c->hDT[L], nullptr);
  rop_h(c, B, nullptr);
  for (int l = L; l >= 1; --l) rbackward_h(c, l, B, mode, true, out, nullptr);
}

// ------------------------------------------------ precision dispatch
// Narrow nets: the solve's cache also copied into the concatenated columns of
// the weight-gradient GEMM (X and A_1 .. A_{L-1}; for the Hessian delta_2 ..
// delta_L), when the narrow product will serve this batch.
void narrow_cache(hf_ctx* c, const float* X, int B, bool hess) {
  c->cat_B = -1;
  const int L = c->L;
  if (!c->narrow_cat || B > c->Bws || !narrow_eligible(L, c->d.data(), X, nullptr) ||
      gemm_tile(B, c->d[1], c->d[0]) != 64)
    return;
  NarrowGather g;
  std::memset(&g, 0, sizeof g);
  g.B = B;
  g.ldd[0] = c->ldy_cat;
  g.ldd[1] = c->ldr_cat;
  int k = 0;
  for (int l = 0; l < L; ++l) {
    g.src[k] = l == 0 ? X : c->F(c->oA[l]);
    g.lds[k] = l == 0 ? c->d[0] : c->ld[l];
    g.cols[k] = c->d[l];
    g.dst[k] = c->F(c->oYcat) + c->yoff[l];
    g.which[k] = 0;
    ++k;
  }
  if (hess) {
    for (int l = 2; l <= L; ++l) {
      g.src[k] = c->F(c->oD[l]);
      g.lds[k] = c->ld[l];
      g.cols[k] = c->d[l];
      g.dst[k] = c->F(c->oDcat) + c->roff[l];
      g.which[k] = 1;
      ++k;
    }
  }
  g.nblk = k;
  narrow_gather(c->launch(), g);
  c->cat_B = B;
  c->cat_hess = hess;
}

// Whether the cache of a narrow net is built by the narrow kernels: the
// products that follow must take a narrow form (every vector they multiply
// is aligned: the solvers' own, or v_ext, the caller's x0 or v, which may be
// null), since the narrow build leaves the transposed weights of the GEMM
// path unwritten.
bool narrow_build_ok(const hf_ctx* c, const float* X, const float* v_ext, int B) {
  return c->narrow_cat && B <= c->Bws && narrow_eligible(c->L, c->d.data(), X, v_ext) &&
         narrow_eligible(c->L, c->d.data(), nullptr, c->F(c->oPv)) &&
         gemm_tile(B, c->d[1], c->d[0]) == 64;
}

// What narrow_build forms: the cache of a solve; the gradient's pass (loss
// partials into oLoss, delta_1 .. delta_L into the concatenated columns); or
// the loss alone (partials into oLoss).  After either of the last two no
// solve's cache is held.
enum NarrowPass { NARROW_CACHE, NARROW_GRAD, NARROW_LOSS };

void narrow_build(hf_ctx* c, const float* W, const float* X, int B,
                  const int32_t* y, bool hess, NarrowPass pass = NARROW_CACHE) {
  const bool grad = pass == NARROW_GRAD, loss = pass != NARROW_CACHE;
  const int L = c->L;
  c->cat_B = -1;
  NarrowFwdArgs a;
  std::memset(&a, 0, sizeof a);
  a.L = L;
  a.B = B;
  a.act = c->act;
  a.hess = hess ? 1 : 0;
  for (int l = 0; l <= L; ++l) {
    a.d[l] = c->d[l];
    a.ld[l] = l == 0 ? c->d[0] : c->ld[l];
    a.offW[l] = l == 0 ? 0 : (long long)c->offW[l];
    a.offB[l] = l == 0 ? 0 : (long long)c->offB[l];
    if (l >= 1 && l < L) {
      a.A[l] = c->F(c->oA[l]);
      a.E2[l] = c->F(c->oE2[l]);
    }
    if (l >= 2) a.D[l] = c->F(c->oD[l]);
    a.yoff[l] = c->yoff[l];
    a.roff[l] = c->roff[l];
  }
  a.X = X;
  a.W = W;
  a.y = hess || loss ? y : nullptr;
  a.P = loss ? nullptr : c->F(c->oP);
  a.Ycat = pass == NARROW_LOSS ? nullptr : c->F(c->oYcat);
  a.ldy = c->ldy_cat;
  a.Dcat = hess || grad ? c->F(c->oDcat) : nullptr;
  a.ldr = c->ldr_cat;
  a.invB = 1.0f / (float)B;
  a.err = c->errp();
  a.grad = grad ? 1 : 0;
  a.loss_part = loss ? c->Dp(c->oLoss) : nullptr;
  narrow_forward(c->launch(), a);
  if (!loss) {
    c->cat_B = B;
    c->cat_hess = hess;
  }
}

// The cache of a solve on the curvature batch: forward pass, p and, for the
// Hessian, delta_l and (delta_l W_l) phi''(A_{l-1}).
void build_cache(hf_ctx* c, const float* W, const float* X, int B,
                 const int32_t* y, bool hess, const float* v_ext = nullptr) {
  if (c->bf16()) {
    forward_plain_h(c, W, X, B, hess ? y : nullptr, hess);
    if (hess)
      for (int l = c->L; l >= 2; --l) backward_data_h(c, l, B, true);
  } else if (narrow_build_ok(c, X, v_ext, B)) {
    narrow_build(c, W, X, B, y, hess);
  } else {
    forward_plain(c, W, X, B, hess ? y : nullptr, hess);
    if (hess)
      for (int l = c->L; l >= 2; --l) backward_data(c, W, l, B, true);
    narrow_cache(c, X, B, hess);
  }
}

void product(hf_ctx* c, const float* W, const float* X, int B, const float* v,
             int mode, float* out, const int* skip) {
  if (c->bf16()) product_cached_h(c, B, v, mode, out, skip);
  else product_cached(c, W, X, B, v, mode, out, skip);
}

// A CG iteration's product q = A p (skipped once the solve has stopped);
// where the product's last kernel can also form the partials of p.q and p.p
// for the iteration's update, it does, and the count of partials is
// returned (0: the iteration's dot kernel forms them).
int product_cg(hf_ctx* c, const float* W, const float* X, int B, const float* p,
               int mode, float* q, double* part, CgState* st, int j) {
  c->fuse = {p, part, st, j};
  c->fused_blocks = 0;
  product(c, W, X, B, p, mode, q, &st->done);
  c->fuse = {};
  const int fb = c->fused_blocks;
  c->fused_blocks = 0;
  return fb;
}

// q += lambda v: the damping term of B_k = A + lambda I (Alg. 1 step 3)
void lambda_axpy(hf_ctx* c, float* q, const float* v, float lambda,
                 const int* skip) {
  if (lambda != 0.0f) axpy(c->launch(), q, v, lambda, c->n, skip);
}

}  // namespace

namespace {

// f on B rows (forward pass only) into loss (fp32) and/or loss64 (fp64)
void loss_only(hf_ctx* c, const float* W, const float* X, const int32_t* y,
               int B, float* loss, double* loss64) {
  if (c->bf16()) forward_plain_h(c, W, X, B, y, false);
  else if (narrow_build_ok(c, X, nullptr, B)) narrow_build(c, W, X, B, y, false, NARROW_LOSS);
  else forward_plain(c, W, X, B, y, false);
  loss_finalize(c->launch(), c->Dp(c->oLoss), (B + 3) / 4, B, loss, loss64);
}

// f and g on B rows (arguments already checked).  With `fisher` the same
// backward pass also forms F = (1/B) sum_b grad l_b^2: delta_l carries the
// 1/B of the mean, so the squared-operand weight gradient
// B sum_b delta_l^2 a_{l-1}^2 is F's weight block, and B sum_b delta_l^2
// its bias block.  bf16 contexts square the two transposed operands in
// place once the gradient has read them (the backward step reads the
// row-major copies), then run the same weight-gradient GEMM again.
void loss_grad_any(hf_ctx* c, const float* W, const float* X, const int32_t* y,
                   int b, float* loss, double* loss64, float* grad,
                   float* fisher = nullptr) {
  if (c->bf16()) {
    forward_plain_h(c, W, X, b, y, true);
    loss_finalize(c->launch(), c->Dp(c->oLoss), (b + 3) / 4, b, loss, loss64);
    for (int l = c->L; l >= 1; --l) {
      bf16_t* dT = c->H(c->hDT[l]);
      bf16_t* aT = c->H(l == 1 ? c->hXT : c->hAT[l - 1]);
      wgrad_h(c, l, b, dT, aT, nullptr, nullptr, grad, nullptr);
      if (fisher) {
        square_bf16(c->launch(), dT, (long long)c->d[l] * c->ldB);
        square_bf16(c->launch(), aT, (long long)c->d[l - 1] * c->ldB);
        wgrad_h(c, l, b, dT, aT, nullptr, nullptr, fisher, nullptr);
      }
      if (l > 1) backward_data_h(c, l, b, false);
    }
    if (fisher) waxpy(c->launch(), fisher, nullptr, (double)b, fisher, c->n);
    return;
  }
  if (!fisher && narrow_build_ok(c, X, nullptr, b)) {
    // narrow nets: the forward and backward pass in two launches, then every
    // layer's gradient from one GEMM over the concatenated columns
    narrow_build(c, W, X, b, y, false, NARROW_GRAD);
    loss_finalize(c->launch(), c->Dp(c->oLoss), (b + 3) / 4, b, loss, loss64);
    cat_wgrad(c, b, c->F(c->oDcat), nullptr, nullptr, grad, nullptr, nullptr);
    return;
  }
  forward_plain(c, W, X, b, y, true);
  loss_finalize(c->launch(), c->Dp(c->oLoss), (b + 3) / 4, b, loss, loss64);
  for (int l = c->L; l >= 1; --l) {
    const float* Ain = (l == 1) ? X : c->F(c->oA[l - 1]);
    const int ldin = (l == 1) ? c->d[0] : c->ld[l - 1];
    wgrad(c, l, b, c->F(c->oD[l]), Ain, nullptr, nullptr, ldin, grad, nullptr);
    if (fisher)
      wgrad(c, l, b, c->F(c->oD[l]), Ain, nullptr, nullptr, ldin, fisher,
            nullptr, true);
    if (l > 1) backward_data(c, W, l, b, false);
  }
  if (fisher) waxpy(c->launch(), fisher, nullptr, (double)b, fisher, c->n);
}

}  // namespace

namespace {

// Iterates kept for CG-backtracking: after j solver updates for every j of
// the schedule (j = 1, then j <- max(j + 1, ceil(13 j / 10)), j < max_iters,
// the latest `cap` of them), each into its own vector of buf.  A copy
// enqueued after the solve has stopped does nothing (device flag).
struct KeepPlan {
  std::vector<int> js;   // increasing
  float* buf = nullptr;
  KeepPlan(int max_iters, int cap, float* b) : buf(b) {
    for (int j = 1; j < max_iters; j = std::max(j + 1, (13 * j + 9) / 10))
      js.push_back(j);
    if ((int)js.size() > cap) js.erase(js.begin(), js.end() - cap);
  }
  // slot of iteration count j, or -1
  int slot(int j) const {
    for (size_t i = 0; i < js.size(); ++i)
      if (js[i] == j) return (int)i;
    return -1;
  }
  void after(const Launch& L, int j, const float* x, long long n,
             const int* skip) const {
    const int i = slot(j);
    if (i >= 0) keep_iterate(L, buf + (size_t)i * n, x, n, skip);
  }
};

// CG iterations per captured graph.  Each graph launch costs the GPU about
// 13 us between the last kernel of one replay and the first of the next; on
// the 784-100-10 net (iterations of about 45 us of kernels) five
// Gauss-Newton iterations per graph took its 10-iteration solve from 634 to
// 563 us.  Hessian solves usually stop at a detection within a few
// iterations, and the iterations captured past the stop would be launched
// for nothing: one per graph.
int cg_graph_iters(int mode) { return mode == HF_HESSIAN ? 1 : 5; }

// Make c->cg_exec replay cg_graph_iters(mode) CG iterations with these
// arguments: each the cached product q = A p and the vector kernels, with
// the iteration index kept on
// the device and the stop flag written to host-pinned memory.  Returns
// false (and switches graphs off for the context) if the capture fails;
// the caller then runs the launch-by-launch loop.
bool cg_graph(hf_ctx* c, const float* W, const float* Xc, int b, const float* g,
              float* step, float* neg_dir, int mode, const float* minv) {
  const hf_ctx::CgKey key = {W, Xc, g, step, neg_dir, minv, c->ws, b, c->Bws, mode};
  if (c->cg_exec && c->cg_key == key) return true;
  if (c->cg_exec) {
    (void)hipGraphExecDestroy(c->cg_exec);
    c->cg_exec = nullptr;
  }
  auto off = [&]() {
    c->graphs_off = true;
    (void)hipGetLastError();
    return false;
  };
  if (!c->cap_stream &&
      hipStreamCreateWithFlags(&c->cap_stream, hipStreamNonBlocking) != hipSuccess)
    return off();
  if (!c->hflag) {
    if (hipHostMalloc((void**)&c->hflag, 64, hipHostMallocMapped | hipHostMallocCoherent) !=
        hipSuccess) {
      c->hflag = nullptr;
      return off();
    }
    if (hipHostGetDevicePointer((void**)&c->hflag_dev, c->hflag, 0) != hipSuccess ||
        !c->hflag_dev)
      return off();
  }
  CgState* st = reinterpret_cast<CgState*>(c->ws + c->oState);
  const hipStream_t user = c->stream;
  if (hipStreamBeginCapture(c->cap_stream, hipStreamCaptureModeRelaxed) != hipSuccess)
    return off();
  c->stream = c->cap_stream;
  // only the graph's last iteration stores the stop flag in host memory
  // (its direction kernel stores it whether or not the solve stopped
  // earlier in the graph); a store there delays the next kernel's start
  const int K = cg_graph_iters(mode);
  for (int k = 0; k < K; ++k) {
    const int fb = product_cg(c, W, Xc, b, c->F(c->oPv), mode, c->F(c->oQ), c->Dp(c->oRed), st,
                              -1);
    cg_iteration(c->launch(), step, c->F(c->oR), c->F(c->oPv), c->F(c->oQ), g, neg_dir,
                 c->n, -1, c->Dp(c->oRed), st, minv, k == K - 1 ? c->hflag_dev : nullptr, fb);
  }
  c->stream = user;
  hipGraph_t graph = nullptr;
  const hipError_t e1 = hipStreamEndCapture(c->cap_stream, &graph);
  if (e1 != hipSuccess || !graph) return off();
  const hipError_t e2 = hipGraphInstantiate(&c->cg_exec, graph, nullptr, nullptr, 0);
  (void)hipGraphDestroy(graph);
  if (e2 != hipSuccess) {
    c->cg_exec = nullptr;
    return off();
  }
  c->cg_key = key;
  return true;
}

// CG-Minimize after argument checks; x0 (device, may be null) is the warm
// start of Alg. 2
int solve_cg(hf_ctx* c, const float* W, const float* Xc, const int32_t* yc,
             int b, const float* g, float damping, int32_t max_iters,
             float rel_tol, int32_t mode, const float* x0, float* step,
             float* neg_dir, hf_cg_info* info, const KeepPlan* keep = nullptr,
             const float* minv = nullptr) {
  std::memset(info, 0, sizeof *info);
  if (!c->pinned) {
    HIP_TRY(c, hipHostMalloc((void**)&c->pinned, 2 * sizeof(CgState), hipHostMallocDefault));
    for (auto& e : c->ev) HIP_TRY(c, hipEventCreateWithFlags(&e, hipEventDisableTiming));
  }
  if (c->prof) c->prof->solve_begin = c->prof->pending.size();
  const Launch Lc = c->launch();
  const long long n = c->n;
  const bool hess = mode == HF_HESSIAN;
  CgState* st = reinterpret_cast<CgState*>(c->ws + c->oState);
  const int* skip = &st->done;
  double* part = c->Dp(c->oRed);
  float* r = c->F(c->oR);
  float* p = c->F(c->oPv);
  float* q = c->F(c->oQ);

  // cache of the curvature batch: activations, p, delta_l, E2_l
  build_cache(c, W, Xc, b, yc, hess, x0);
  // a warm start's residual needs one product on the cache
  const int k0 = x0 ? 1 : 0;
  if (x0) {
    product(c, W, Xc, b, x0, mode, q, nullptr);
    trace_product(c, 0, x0, q, nullptr);
  }
  cg_init(Lc, g, x0, x0 ? q : nullptr, step, r, p, neg_dir, n, (double)damping,
          (double)rel_tol * (double)rel_tol, part, st, minv, max_iters);
  // Replay captured iterations when nothing needs per-iteration host work
  // (kernel timing, kept iterates, the product trace): one graph launch per
  // cg_graph_iters(mode) iterations instead of a launch per kernel.  The
  // device also stops the solve at the budget, so that nothing replayed past
  // it does any work.
  const bool replay = max_iters > 0 && !c->prof && !keep && !c->trace_buf &&
                      !c->graphs_off &&
                      cg_graph(c, W, Xc, b, g, step, neg_dir, mode, minv);
  if (replay) {
    *(volatile int*)c->hflag = 0;
    const int K = cg_graph_iters(mode);
    const int launches = (max_iters + K - 1) / K;
    for (int j = 0; j < launches; ++j) {
      HIP_TRY(c, hipGraphLaunch(c->cg_exec, c->stream));
      HIP_TRY(c, hipEventRecord(c->ev[j & 1], c->stream));
      if (j >= 1) {
        HIP_TRY(c, hipEventSynchronize(c->ev[(j - 1) & 1]));
        if (*(volatile int*)c->hflag) break;
      }
    }
  }
  for (int j = 0; !replay && j < max_iters; ++j) {
    if (c->prof) c->prof->tag = j;
    const int fb = product_cg(c, W, Xc, b, p, mode, q, part, st, j);
    trace_product(c, k0 + j, p, q, skip);
    cg_iteration(Lc, step, r, p, q, g, neg_dir, n, j, part, st, minv, nullptr, fb);
    if (keep) keep->after(Lc, j + 1, step, n, skip);
    // Stop enqueueing once the device reports `done` for the previous
    // iteration; the work already queued for this one returns at once.
    HIP_TRY(c, hipMemcpyAsync(&c->pinned[j & 1], st, sizeof(CgState),
                              hipMemcpyDeviceToHost, c->stream));
    HIP_TRY(c, hipEventRecord(c->ev[j & 1], c->stream));
    if (j >= 1) {
      HIP_TRY(c, hipEventSynchronize(c->ev[(j - 1) & 1]));
      if (c->pinned[(j - 1) & 1].done) break;
    }
  }
  if (c->prof) c->prof->tag = -1;
  HIP_TRY(c, hipGetLastError());
  HIP_TRY(c, hipMemcpyAsync(&c->pinned[0], st, sizeof(CgState),
                            hipMemcpyDeviceToHost, c->stream));
  int errflag = 0;
  HIP_TRY(c, hipMemcpyAsync(&errflag, c->ws + c->oErr, sizeof(int),
                            hipMemcpyDeviceToHost, c->stream));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  const CgState& s = c->pinned[0];
  if (c->prof)
    c->prof->retract(s.products - 1, s.neg || (s.status && s.iters < s.products),
                     s.neg ? s.neg_iter : -1);
  info->iters = s.iters;
  info->products = s.products + (x0 ? 1 : 0);
  info->neg_curv = s.neg;
  info->neg_iter = s.neg ? s.neg_iter : -1;
  info->pBp = s.neg ? s.kappa : 0.0;
  info->pHp = s.neg ? s.pq : 0.0;
  info->gTd = s.neg ? (s.gp >= 0.0 ? -s.gp : s.gp) : 0.0;
  info->rr0 = s.rr0;
  info->rr_final = s.rr[s.iters & 1];
  info->status = s.status;
  info->replayed = replay ? 1 : 0;
  if (errflag) {
    info->status = HF_ELABEL;
    int zero = 0;
    HIP_TRY(c, hipMemcpy(c->ws + c->oErr, &zero, sizeof(int), hipMemcpyHostToDevice));
    return fail(c, HF_ELABEL, "a label outside [0, %d) was seen", c->d[c->L]);
  }
  if (s.status) return fail(c, HF_ENUMERIC, "non-finite CG scalar");
  return HF_OK;
}

// Bi-CG-STAB after argument checks; x0 (device, may be null) is the warm
// start of Alg. 2; minv (device, may be null) the diagonal of M^-1 of a
// solve preconditioned on the right
int solve_bicg(hf_ctx* c, const float* W, const float* Xc, const int32_t* yc,
               int b, const float* g, float damping, int32_t max_iters,
               float rel_tol, int32_t mode, const float* x0, float* step,
               float* neg_dir, hf_cg_info* info, const KeepPlan* keep = nullptr,
               const float* minv = nullptr) {
  std::memset(info, 0, sizeof *info);
  if (!c->pinned) {
    HIP_TRY(c, hipHostMalloc((void**)&c->pinned, 2 * sizeof(CgState), hipHostMallocDefault));
    for (auto& e : c->ev) HIP_TRY(c, hipEventCreateWithFlags(&e, hipEventDisableTiming));
  }
  BicgState* hostst = reinterpret_cast<BicgState*>(c->pinned_bicg);
  if (!hostst) {
    HIP_TRY(c, hipHostMalloc((void**)&c->pinned_bicg, 2 * sizeof(BicgState),
                             hipHostMallocDefault));
    hostst = reinterpret_cast<BicgState*>(c->pinned_bicg);
  }
  if (c->prof) c->prof->solve_begin = c->prof->pending.size();
  const Launch Lc = c->launch();
  const long long n = c->n;
  const bool hess = mode == HF_HESSIAN;
  BicgState* st = reinterpret_cast<BicgState*>(c->ws + c->oState);
  const int* skip = &st->done;
  double* part = c->Dp(c->oRed);
  float* r = c->F(c->oR);
  float* p = c->F(c->oPv);
  float* Ap = c->F(c->oQ);
  float* sv = c->F(c->oS);
  float* t = c->F(c->oT);
  float* rs = c->F(c->oRs);
  // the vectors the products are taken of
  float* ph = minv ? c->F(c->oPh) : p;
  float* sh = minv ? c->F(c->oSh) : sv;

  build_cache(c, W, Xc, b, yc, hess, x0);
  // a warm start's residual needs one product on the cache
  const int k0 = x0 ? 1 : 0;
  if (x0) {
    product(c, W, Xc, b, x0, mode, Ap, nullptr);
    trace_product(c, 0, x0, Ap, nullptr);
  }
  bicg_init(Lc, g, x0, x0 ? Ap : nullptr, step, r, rs, p, neg_dir, n,
            (double)damping, (double)rel_tol * (double)rel_tol, part, st, minv,
            ph);
  for (int j = 0; j < max_iters; ++j) {
    if (c->prof) c->prof->tag = 2 * j;
    product(c, W, Xc, b, ph, mode, Ap, skip);
    trace_product(c, k0 + 2 * j, ph, Ap, skip);
    lambda_axpy(c, Ap, ph, damping, skip);
    bicg_half(Lc, r, rs, Ap, sv, n, j, part, st, minv, sh);
    if (c->prof) c->prof->tag = 2 * j + 1;
    product(c, W, Xc, b, sh, mode, t, skip);
    trace_product(c, k0 + 2 * j + 1, sh, t, skip);
    lambda_axpy(c, t, sh, damping, skip);
    bicg_rest(Lc, step, r, rs, p, Ap, sv, t, g, neg_dir, n, j, part, st, minv,
              ph, sh);
    if (keep) keep->after(Lc, j + 1, step, n, skip);
    HIP_TRY(c, hipMemcpyAsync(&hostst[j & 1], st, sizeof(BicgState),
                              hipMemcpyDeviceToHost, c->stream));
    HIP_TRY(c, hipEventRecord(c->ev[j & 1], c->stream));
    if (j >= 1) {
      HIP_TRY(c, hipEventSynchronize(c->ev[(j - 1) & 1]));
      if (hostst[(j - 1) & 1].done) break;
    }
  }
  if (c->prof) c->prof->tag = -1;
  HIP_TRY(c, hipGetLastError());
  HIP_TRY(c, hipMemcpyAsync(&hostst[0], st, sizeof(BicgState),
                            hipMemcpyDeviceToHost, c->stream));
  int errflag = 0;
  HIP_TRY(c, hipMemcpyAsync(&errflag, c->ws + c->oErr, sizeof(int),
                            hipMemcpyDeviceToHost, c->stream));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  const BicgState& s = hostst[0];
  if (c->prof) c->prof->retract_bicg(s.products, s.neg ? s.neg_iter : -1);
  info->iters = s.iters;
  info->products = s.products + (x0 ? 1 : 0);
  info->neg_curv = s.neg;
  info->neg_iter = s.neg ? s.neg_iter : -1;
  info->pBp = s.neg ? s.dBd : 0.0;
  info->pHp = s.neg ? s.dHd : 0.0;
  info->gTd = s.neg ? s.gTd : 0.0;
  info->rr0 = s.rr0;
  info->rr_final = s.rr;
  info->status = s.status;
  if (errflag) {
    info->status = HF_ELABEL;
    int zero = 0;
    HIP_TRY(c, hipMemcpy(c->ws + c->oErr, &zero, sizeof(int), hipMemcpyHostToDevice));
    return fail(c, HF_ELABEL, "a label outside [0, %d) was seen", c->d[c->L]);
  }
  if (s.status) return fail(c, HF_ENUMERIC, "non-finite Bi-CG-STAB scalar");
  return HF_OK;
}

}  // namespace

namespace {

// Stateless product out = A v on B rows (arguments already checked).
void hvp_any(hf_ctx* c, const float* W, const float* X, const int32_t* y, int b,
             const float* v, int mode, float* out) {
  const Launch Lc = c->launch();
  const int L = c->L;
  if (c->bf16()) {
    // Large batches: the forward pass of a solve, then its product, whose
    // single-product GEMMs take 256 x 256 tiles, instead of the fused
    // forward / R-forward and backward / R-backward kernels (128 x 128
    // tiles), once the 256 x 256 tiles of the first layer cover the 256 CUs
    // (speech net at 16,384 rows: Hv 7.0 -> 6.0 ms, Gv 4.4 -> 3.7 ms).
    if (c->cached_layout && (long long)(b / 256) * (c->d[1] / 256) >= 256) {
      build_cache(c, W, X, b, y, mode == HF_HESSIAN, v);
      product(c, W, X, b, v, mode, out, nullptr);
      return;
    }
    hvp_h(c, W, X, y, b, v, mode, out);
    return;
  }
  // Small batch-row GEMMs: the fused forward / R-forward and backward /
  // R-backward kernels below have only 128 x 128 tiles and no split K, so a
  // grid of fewer than 128 workgroups (half the compute units) would run
  // long K chains on a few units.  The cached route (the forward pass of a
  // solve, then its product) takes 64 x 64 tiles and split K there.
  if (c->cached_layout &&
      (long long)((b + 127) / 128) * ((c->d[1] + 127) / 128) < 128) {
    build_cache(c, W, X, b, y, mode == HF_HESSIAN, v);
    product_cached(c, W, X, b, v, mode, out, nullptr);
    return;
  }
  c->cat_B = -1;
  // forward fused with R-forward
  for (int l = 1; l <= L; ++l) {
    GemmShape s;
    if (l == 1) {
      s = shape(b, c->d[1], c->d[0], X, nullptr, W + c->offW[1], v + c->offW[1],
                c->d[0], c->d[0], 1, nullptr);
    } else {
      s = shape(b, c->d[l], c->d[l - 1], c->F(c->oA[l - 1]), c->F(c->oRA[l - 1]),
                W + c->offW[l], v + c->offW[l], c->ld[l - 1], c->d[l - 1], 1,
                nullptr);
    }
    EpiArgs e = epi(c, l < L);
    e.bias = W + c->offB[l];
    e.rbias = v + c->offB[l];
    e.out0 = (l < L) ? c->F(c->oA[l]) : c->F(c->oZ);
    e.out1 = c->F(c->oRZ[l]);
    e.out2 = (l < L) ? c->F(c->oRA[l]) : nullptr;
    e.ldo = c->ld[l];
    gemm_fwd_rfwd(Lc, s, e);
  }
  const bool hess = mode == HF_HESSIAN;
  softmax_xent(Lc, c->F(c->oZ), hess ? y : nullptr, b, c->d[L], c->ld[L],
               c->F(c->oP), hess ? c->F(c->oD[L]) : nullptr, c->Dp(c->oLoss),
               c->errp());
  softmax_rop(Lc, c->F(c->oP), c->F(c->oRZ[L]), b, c->d[L], c->ld[L],
              c->F(c->oRD[L]), nullptr);
  for (int l = L; l >= 1; --l) {
    const float* Ain = (l == 1) ? X : c->F(c->oA[l - 1]);
    const int ldin = (l == 1) ? c->d[0] : c->ld[l - 1];
    if (hess && l > 1) {
      wgrad(c, l, b, c->F(c->oRD[l]), Ain, c->F(c->oD[l]), c->F(c->oRA[l - 1]),
            ldin, out, nullptr);
    } else {
      wgrad(c, l, b, c->F(c->oRD[l]), Ain, nullptr, nullptr, ldin, out, nullptr);
    }
    if (l == 1) break;
    EpiArgs e = epi(c, 1);
    e.ldo = c->ld[l - 1];
    e.aux0 = c->F(c->oA[l - 1]);
    e.lda = c->ld[l - 1];
    if (hess) {
      // (E, RE) = (delta W, Rdelta W + delta V) in one pass
      GemmShape s = shape(b, c->d[l - 1], c->d[l], c->F(c->oD[l]), c->F(c->oRD[l]),
                          W + c->offW[l], v + c->offW[l], c->ld[l], c->d[l - 1],
                          1, nullptr);
      e.out0 = c->F(c->oD[l - 1]);
      e.out1 = c->F(c->oRD[l - 1]);
      e.aux1 = c->F(c->oRZ[l - 1]);
      gemm_bwd_rbwd(Lc, s, e);
    } else {
      GemmShape s = shape(b, c->d[l - 1], c->d[l], c->F(c->oRD[l]), nullptr,
                          W + c->offW[l], nullptr, c->ld[l], c->d[l - 1], 1,
                          nullptr);
      e.out1 = c->F(c->oRD[l - 1]);
      gemm_gnbwd(Lc, s, e);
    }
  }
}

}  // namespace

// ==================================================================== C ABI
extern "C" {

int hf_create(const int32_t* dims, int32_t n_dims, int32_t act, int32_t prec,
              int64_t max_batch, void* hip_stream, hf_ctx** out) {
  if (!out) return HF_EINVAL;
  *out = nullptr;
  if (!dims || n_dims < 2 || n_dims > HF_MAX_LAYERS + 1) return HF_EINVAL;
  if (!valid_act(act) || (prec != HF_FP32 && prec != HF_BF16_INPUTS) || max_batch < 1)
    return HF_EINVAL;
  for (int i = 0; i < n_dims; ++i)
    if (dims[i] < 1) return HF_EINVAL;
  if (dims[n_dims - 1] > HF_MAX_CLASSES) return HF_EINVAL;
  const int64_t lim = (int64_t(1) << 31) - 1;
  int64_t n = 0;
  for (int i = 0; i < n_dims; ++i)
    if (((max_batch + 255) & ~int64_t(255)) * (int64_t)round64(dims[i]) > lim ||
        ((max_batch + 63) & ~int64_t(63)) * (int64_t)round256(dims[i]) > lim)
      return HF_EINVAL;
  for (int l = 1; l < n_dims; ++l) n += (int64_t)dims[l] * (dims[l - 1] + 1);
  if (n > lim - 64) return HF_EINVAL;
  hf_ctx* c = new (std::nothrow) hf_ctx();
  if (!c) return HF_ENOMEM;
  c->L = n_dims - 1;
  c->d.assign(dims, dims + n_dims);
  c->ld.resize(n_dims);
  for (int i = 0; i < n_dims; ++i) c->ld[i] = round4(dims[i]);
  c->ldh.resize(n_dims);
  for (int i = 0; i < n_dims; ++i) c->ldh[i] = round64(dims[i]);
  c->act = act;
  c->prec = prec;
  c->Bmax = max_batch;
  c->n = n;
  c->offW.assign(n_dims, 0);
  c->offB.assign(n_dims, 0);
  int64_t off = 0;
  for (int l = 1; l < n_dims; ++l) {
    c->offW[l] = off;
    off += (int64_t)dims[l] * dims[l - 1];
    c->offB[l] = off;
    off += dims[l];
  }
  c->stream = reinterpret_cast<hipStream_t>(hip_stream);
  plan(c, max_batch);
  *out = c;
  return HF_OK;
}

int hf_destroy(hf_ctx* c) {
  if (!c) return HF_OK;
  delete c->prof;
  delete c->na;
  if (c->cg_exec) (void)hipGraphExecDestroy(c->cg_exec);
  if (c->cap_stream) (void)hipStreamDestroy(c->cap_stream);
  if (c->hflag) (void)hipHostFree(c->hflag);
  if (c->pinned) (void)hipHostFree(c->pinned);
  if (c->pinned_bicg) (void)hipHostFree(c->pinned_bicg);
  for (auto& e : c->ev)
    if (e) (void)hipEventDestroy(e);
  delete c;
  return HF_OK;
}

int hf_set_stream(hf_ctx* c, void* s) {
  if (!c) return HF_EINVAL;
  c->stream = reinterpret_cast<hipStream_t>(s);
  return HF_OK;
}

int64_t hf_num_params(const hf_ctx* c) { return c ? c->n : -1; }

size_t hf_workspace_bytes(const hf_ctx* c, int64_t batch) {
  if (!c) return 0;
  if (batch <= 0) batch = c->Bmax;
  if (batch > c->Bmax) return 0;
  return plan_bytes(c, batch);
}

int hf_set_workspace(hf_ctx* c, void* p, size_t bytes) {
  if (!c) return HF_EINVAL;
  if (!p) return fail(c, HF_EINVAL, "workspace pointer is NULL");
  if ((uintptr_t)p & 255u) return fail(c, HF_EINVAL, "workspace is not 256-byte aligned");
  const size_t need1 = plan_bytes(c, 1);
  if (bytes < need1)
    return fail(c, HF_EWORKSPACE, "workspace of %zu bytes is smaller than the %zu needed "
                "for one row", bytes, need1);
  // the largest batch whose layout fits (the bytes needed grow with the batch)
  int64_t lo = 1, hi = c->Bmax;
  while (lo < hi) {
    const int64_t mid = lo + (hi - lo + 1) / 2;
    if (plan_bytes(c, mid) <= bytes) lo = mid;
    else hi = mid - 1;
  }
  c->ws = nullptr;
  plan(c, lo);
  c->ws = reinterpret_cast<char*>(p);
  c->ws_bytes = bytes;
  HIP_TRY(c, hipMemset(c->ws + c->oErr, 0, sizeof(int)));
  // bf16 operands: the zeros in their padding columns are never rewritten;
  // nor are the zero blocks of the narrow nets' concatenated delta and RA
  // columns (layer 1 has no second weight-gradient term); wait for the fills
  // so that no later stream can run ahead of them
  if (c->hend > c->hbeg) HIP_TRY(c, hipMemset(c->ws + c->hbeg, 0, c->hend - c->hbeg));
  if (c->narrow_cat) {
    HIP_TRY(c, hipMemset(c->ws + c->oRAcat, 0, (size_t)c->Bws * c->ldy_cat * sizeof(float)));
    HIP_TRY(c, hipMemset(c->ws + c->oDcat, 0, (size_t)c->Bws * c->ldr_cat * sizeof(float)));
  }
  if (c->hend > c->hbeg || c->narrow_cat) HIP_TRY(c, hipDeviceSynchronize());
  return HF_OK;
}

int hf_loss_grad(hf_ctx* c, const float* W, const float* X, const int32_t* y,
                 int64_t B, float* loss, float* grad) {
  int rc;
  if ((rc = check_ready(c))) return rc;
  if ((rc = check_ptr(c, W, "W")) || (rc = check_ptr(c, X, "X")) ||
      (rc = check_ptr(c, grad, "grad")) || (rc = check_batch(c, B)))
    return rc;
  if (!y) return fail(c, HF_EINVAL, "y is NULL");
  if (!loss) return fail(c, HF_EINVAL, "loss is NULL");
  loss_grad_any(c, W, X, y, (int)B, loss, nullptr, grad);
  HIP_TRY(c, hipGetLastError());
  return HF_OK;
}

int hf_loss(hf_ctx* c, const float* W, const float* X, const int32_t* y,
            int64_t B, float* loss) {
  int rc;
  if ((rc = check_ready(c))) return rc;
  if ((rc = check_ptr(c, W, "W")) || (rc = check_ptr(c, X, "X")) ||
      (rc = check_batch(c, B)))
    return rc;
  if (!y) return fail(c, HF_EINVAL, "y is NULL");
  if (!loss) return fail(c, HF_EINVAL, "loss is NULL");
  loss_only(c, W, X, y, (int)B, loss, nullptr);
  HIP_TRY(c, hipGetLastError());
  return HF_OK;
}

int hf_hvp(hf_ctx* c, const float* W, const float* X, const int32_t* y,
           int64_t B, const float* v, int32_t mode, float* out) {
  int rc;
  if ((rc = check_ready(c))) return rc;
  if ((rc = check_ptr(c, W, "W")) || (rc = check_ptr(c, X, "X")) ||
      (rc = check_ptr(c, v, "v")) || (rc = check_ptr(c, out, "out")) ||
      (rc = check_batch(c, B)))
    return rc;
  if (mode != HF_HESSIAN && mode != HF_GAUSS_NEWTON)
    return fail(c, HF_EINVAL, "unknown mode %d", mode);
  if (mode == HF_HESSIAN && !y) return fail(c, HF_EINVAL, "y is NULL");
  hvp_any(c, W, X, y, (int)B, v, mode, out);
  HIP_TRY(c, hipGetLastError());
  return HF_OK;
}

int hf_hvp_noalloc(hf_ctx* c, const float* W, const float* X, const int32_t* y,
                   int64_t B, const float* v, int32_t mode, float* out,
                   int32_t* label_err) {
  int rc;
  if (!c) return HF_EINVAL;
  if ((rc = check_ptr(c, W, "W")) || (rc = check_ptr(c, X, "X")) ||
      (rc = check_ptr(c, v, "v")) || (rc = check_ptr(c, out, "out")))
    return rc;
  if (B < 1 || B > c->Bmax)
    return fail(c, HF_EINVAL, "batch %lld outside [1, %lld]", (long long)B,
                (long long)c->Bmax);
  if (mode != HF_HESSIAN && mode != HF_GAUSS_NEWTON)
    return fail(c, HF_EINVAL, "unknown mode %d", mode);
  if (mode == HF_HESSIAN && !y) return fail(c, HF_EINVAL, "y is NULL");
  if (label_err && ((uintptr_t)label_err & 3u))
    return fail(c, HF_EINVAL, "label_err is not 4-byte aligned");
  const size_t need = plan_bytes(c, B, true);
  if (need > (size_t)HF_NOALLOC_SCRATCH_BYTES)
    return fail(c, HF_EWORKSPACE,
                "%lld rows need %zu bytes of scratch; the no-allocation scratch "
                "holds %zu", (long long)B, need, (size_t)HF_NOALLOC_SCRATCH_BYTES);
  void* base = nullptr;
  HIP_TRY(c, noalloc_scratch(&base));
  if (!c->na) {
    c->na = new (std::nothrow) hf_ctx();
    if (!c->na) return fail(c, HF_ENOMEM, "no host memory for the scratch layout");
    hf_ctx& t = *c->na;
    t.L = c->L;
    t.d = c->d;
    t.ld = c->ld;
    t.ldh = c->ldh;
    t.act = c->act;
    t.prec = c->prec;
    t.Bmax = c->Bmax;
    t.n = c->n;
    t.offW = c->offW;
    t.offB = c->offB;
    t.max_splits = c->max_splits;
  }
  hf_ctx& t = *c->na;
  t.stream = c->stream;
  t.prof = nullptr;
  t.ws = nullptr;
  plan(&t, B, true);
  t.ws = reinterpret_cast<char*>(base);
  t.ws_bytes = HF_NOALLOC_SCRATCH_BYTES;
  t.err_override = label_err;
  // what must start at zero: the label flag and, for bf16 operands, their
  // padding (another call may have left anything there)
  const Launch Lt = t.launch();
  fill_zero(Lt, t.errp(), sizeof(int));
  if (t.hend > t.hbeg) fill_zero(Lt, t.ws + t.hbeg, t.hend - t.hbeg);
  hvp_any(&t, W, X, y, (int)B, v, mode, out);
  HIP_TRY(c, hipGetLastError());
  return HF_OK;
}

int hf_cg(hf_ctx* c, const float* W, const float* Xc, const int32_t* yc,
          int64_t Bc, const float* g, float damping, int32_t max_iters,
          float rel_tol, int32_t mode, float* step, float* neg_dir,
          hf_cg_info* info) {
  int rc;
  if ((rc = check_ready(c))) return rc;
  if ((rc = check_ptr(c, W, "W")) || (rc = check_ptr(c, Xc, "Xc")) ||
      (rc = check_ptr(c, g, "g")) || (rc = check_ptr(c, step, "step")) ||
      (rc = check_ptr(c, neg_dir, "neg_dir")) || (rc = check_batch(c, Bc)))
    return rc;
  if (!info) return fail(c, HF_EINVAL, "info is NULL");
  if (mode != HF_HESSIAN && mode != HF_GAUSS_NEWTON)
    return fail(c, HF_EINVAL, "unknown mode %d", mode);
  if (mode == HF_HESSIAN && !yc) return fail(c, HF_EINVAL, "yc is NULL");
  if (!(damping >= 0.0f) || !std::isfinite(damping))
    return fail(c, HF_EINVAL, "damping must be finite and >= 0");
  if (max_iters < 0) return fail(c, HF_EINVAL, "max_iters < 0");
  if (!(rel_tol >= 0.0f) || !std::isfinite(rel_tol))
    return fail(c, HF_EINVAL, "rel_tol must be finite and >= 0");
  return solve_cg(c, W, Xc, yc, (int)Bc, g, damping, max_iters, rel_tol, mode,
                  nullptr, step, neg_dir, info);
}

int hf_pcg(hf_ctx* c, const float* W, const float* Xc, const int32_t* yc,
           int64_t Bc, const float* g, float damping, int32_t max_iters,
           float rel_tol, int32_t mode, const float* minv, float* step,
           float* neg_dir, hf_cg_info* info) {
  int rc;
  if ((rc = check_ready(c))) return rc;
  if ((rc = check_ptr(c, minv, "minv"))) return rc;
  if ((rc = check_ptr(c, W, "W")) || (rc = check_ptr(c, Xc, "Xc")) ||
      (rc = check_ptr(c, g, "g")) || (rc = check_ptr(c, step, "step")) ||
      (rc = check_ptr(c, neg_dir, "neg_dir")) || (rc = check_batch(c, Bc)))
    return rc;
  if (!info) return fail(c, HF_EINVAL, "info is NULL");
  if (mode != HF_HESSIAN && mode != HF_GAUSS_NEWTON)
    return fail(c, HF_EINVAL, "unknown mode %d", mode);
  if (mode == HF_HESSIAN && !yc) return fail(c, HF_EINVAL, "yc is NULL");
  if (!(damping >= 0.0f) || !std::isfinite(damping))
    return fail(c, HF_EINVAL, "damping must be finite and >= 0");
  if (max_iters < 0) return fail(c, HF_EINVAL, "max_iters < 0");
  if (!(rel_tol >= 0.0f) || !std::isfinite(rel_tol))
    return fail(c, HF_EINVAL, "rel_tol must be finite and >= 0");
  return solve_cg(c, W, Xc, yc, (int)Bc, g, damping, max_iters, rel_tol, mode,
                  nullptr, step, neg_dir, info, nullptr, minv);
}

int hf_fisher_diag(hf_ctx* c, const float* W, const float* X, const int32_t* y,
                   int64_t B, float* out) {
  int rc;
  if ((rc = check_ready(c))) return rc;
  if ((rc = check_ptr(c, W, "W")) || (rc = check_ptr(c, X, "X")) ||
      (rc = check_ptr(c, out, "out")) || (rc = check_batch(c, B)))
    return rc;
  if (!y) return fail(c, HF_EINVAL, "y is NULL");
  // the gradient of the same pass goes to a solver vector no call keeps
  loss_grad_any(c, W, X, y, (int)B, nullptr, nullptr, c->F(c->oT), out);
  HIP_TRY(c, hipGetLastError());
  return HF_OK;
}

int hf_bicgstab(hf_ctx* c, const float* W, const float* Xc, const int32_t* yc,
                int64_t Bc, const float* g, float damping, int32_t max_iters,
                float rel_tol, int32_t mode, float* step, float* neg_dir,
                hf_cg_info* info) {
  int rc;
  if ((rc = check_ready(c))) return rc;
  if ((rc = check_ptr(c, W, "W")) || (rc = check_ptr(c, Xc, "Xc")) ||
      (rc = check_ptr(c, g, "g")) || (rc = check_ptr(c, step, "step")) ||
      (rc = check_ptr(c, neg_dir, "neg_dir")) || (rc = check_batch(c, Bc)))
    return rc;
  if (!info) return fail(c, HF_EINVAL, "info is NULL");
  if (mode != HF_HESSIAN && mode != HF_GAUSS_NEWTON)
    return fail(c, HF_EINVAL, "unknown mode %d", mode);
  if (mode == HF_HESSIAN && !yc) return fail(c, HF_EINVAL, "yc is NULL");
  if (!(damping >= 0.0f) || !std::isfinite(damping))
    return fail(c, HF_EINVAL, "damping must be finite and >= 0");
  if (max_iters < 0) return fail(c, HF_EINVAL, "max_iters < 0");
  if (!(rel_tol >= 0.0f) || !std::isfinite(rel_tol))
    return fail(c, HF_EINVAL, "rel_tol must be finite and >= 0");
  return solve_bicg(c, W, Xc, yc, (int)Bc, g, damping, max_iters, rel_tol,
                    mode, nullptr, step, neg_dir, info);
}

int hf_pbicgstab(hf_ctx* c, const float* W, const float* Xc, const int32_t* yc,
                 int64_t Bc, const float* g, float damping, int32_t max_iters,
                 float rel_tol, int32_t mode, const float* minv, float* step,
                 float* neg_dir, hf_cg_info* info) {
  int rc;
  if ((rc = check_ready(c))) return rc;
  if ((rc = check_ptr(c, minv, "minv"))) return rc;
  if ((rc = check_ptr(c, W, "W")) || (rc = check_ptr(c, Xc, "Xc")) ||
      (rc = check_ptr(c, g, "g")) || (rc = check_ptr(c, step, "step")) ||
      (rc = check_ptr(c, neg_dir, "neg_dir")) || (rc = check_batch(c, Bc)))
    return rc;
  if (!info) return fail(c, HF_EINVAL, "info is NULL");
  if (mode != HF_HESSIAN && mode != HF_GAUSS_NEWTON)
    return fail(c, HF_EINVAL, "unknown mode %d", mode);
  if (mode == HF_HESSIAN && !yc) return fail(c, HF_EINVAL, "yc is NULL");
  if (!(damping >= 0.0f) || !std::isfinite(damping))
    return fail(c, HF_EINVAL, "damping must be finite and >= 0");
  if (max_iters < 0) return fail(c, HF_EINVAL, "max_iters < 0");
  if (!(rel_tol >= 0.0f) || !std::isfinite(rel_tol))
    return fail(c, HF_EINVAL, "rel_tol must be finite and >= 0");
  return solve_bicg(c, W, Xc, yc, (int)Bc, g, damping, max_iters, rel_tol,
                    mode, nullptr, step, neg_dir, info, nullptr, minv);
}

int hf_iterate(hf_ctx* c, float* W, const float* X, const int32_t* y,
               int64_t B, const float* Xc, const int32_t* yc, int64_t Bc,
               const hf_iter_params* prm, int32_t* hybrid_state, float* delta,
               hf_iter_info* info) {
  int rc;
  if ((rc = check_ready(c))) return rc;
  if ((rc = check_ptr(c, W, "W")) || (rc = check_ptr(c, X, "X")) ||
      (rc = check_ptr(c, Xc, "Xc")) || (rc = check_ptr(c, delta, "delta")) ||
      (rc = check_batch(c, B)) || (rc = check_batch(c, Bc)))
    return rc;
  if (!y) return fail(c, HF_EINVAL, "y is NULL");
  if (!prm) return fail(c, HF_EINVAL, "params is NULL");
  if (!info) return fail(c, HF_EINVAL, "info is NULL");
  if (prm->solver != HF_SOLVER_CG && prm->solver != HF_SOLVER_BICGSTAB)
    return fail(c, HF_EINVAL, "unknown solver %d", prm->solver);
  if (prm->curvature != HF_HESSIAN && prm->curvature != HF_GAUSS_NEWTON &&
      prm->curvature != HF_HYBRID)
    return fail(c, HF_EINVAL, "unknown curvature %d", prm->curvature);
  if (prm->curvature == HF_HYBRID && !hybrid_state)
    return fail(c, HF_EINVAL, "hybrid_state is NULL");
  if (prm->curvature != HF_GAUSS_NEWTON && !yc)
    return fail(c, HF_EINVAL, "yc is NULL");
  if (!(prm->damping >= 0.0f) || !std::isfinite(prm->damping))
    return fail(c, HF_EINVAL, "damping must be finite and >= 0");
  if (prm->max_iters < 0) return fail(c, HF_EINVAL, "max_iters < 0");
  if (!(prm->rel_tol >= 0.0f) || !std::isfinite(prm->rel_tol))
    return fail(c, HF_EINVAL, "rel_tol must be finite and >= 0");
  if (!(prm->eta >= 0.0f) || !std::isfinite(prm->eta))
    return fail(c, HF_EINVAL, "eta must be finite and >= 0");
  if (!(prm->armijo_c > 0.0f && prm->armijo_c < 1.0f))
    return fail(c, HF_EINVAL, "armijo_c must lie in (0, 1)");
  if (!(prm->shrink > 0.0f && prm->shrink < 1.0f))
    return fail(c, HF_EINVAL, "shrink must lie in (0, 1)");
  if (prm->max_backtracks < 0) return fail(c, HF_EINVAL, "max_backtracks < 0");
  if (prm->adapt_damping != 0 && prm->adapt_damping != 1)
    return fail(c, HF_EINVAL, "adapt_damping must be 0 or 1");
  if (prm->keep_cap < 0) return fail(c, HF_EINVAL, "keep_cap < 0");
  if (prm->precondition != 0 && prm->precondition != 1)
    return fail(c, HF_EINVAL, "precondition must be 0 or 1");
  if (prm->precondition) {
    if (!(prm->damping > 0.0f))
      return fail(c, HF_EINVAL, "preconditioning needs damping > 0");
    if (!(prm->precond_exp >= 0.0f) || !std::isfinite(prm->precond_exp))
      return fail(c, HF_EINVAL, "precond_exp must be finite and >= 0");
  }
  if (prm->keep_cap > 0 && (rc = check_ptr(c, prm->keep_buf, "keep_buf")))
    return rc;
  std::memset(info, 0, sizeof *info);
  const Launch Lc = c->launch();
  const long long n = c->n;
  const int b = (int)B, bc = (int)Bc;
  float* g = c->F(c->oG);
  float* s = c->F(c->oStep);
  float* d = c->F(c->oNd);
  float* x0v = c->F(c->oX0);
  float* wt = c->F(c->oWt);
  double* scal = c->Dp(c->oScal);       // [0..3] dots, [4] loss
  double hs[5];

  // 1. f_k and g_k on the batch (X, y); with preconditioning the same pass
  // forms the squared per-example gradients F (into the trial weights'
  // vector, free until the line search), and M^-1 = (F + lambda)^-xi
  float* minv = nullptr;
  if (prm->precondition) {
    float* F = wt;
    minv = c->F(c->oMv);
    loss_grad_any(c, W, X, y, b, nullptr, scal + 4, g, F);
    precond_inverse(Lc, F, (double)prm->damping, (double)prm->precond_exp,
                    minv, n);
  } else {
    loss_grad_any(c, W, X, y, b, nullptr, scal + 4, g);
  }
  HIP_TRY(c, hipMemcpyAsync(&hs[4], scal + 4, sizeof(double),
                            hipMemcpyDeviceToHost, c->stream));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  const double f0 = hs[4];
  int errflag = 0;
  HIP_TRY(c, hipMemcpy(&errflag, c->ws + c->oErr, sizeof(int), hipMemcpyDeviceToHost));
  if (errflag) {
    int zero = 0;
    HIP_TRY(c, hipMemcpy(c->ws + c->oErr, &zero, sizeof(int), hipMemcpyHostToDevice));
    return fail(c, HF_ELABEL, "a label outside [0, %d) was seen", c->d[c->L]);
  }
  if (!std::isfinite(f0)) return fail(c, HF_ENUMERIC, "non-finite objective");

  // 2. the curvature of this iteration (Hybrid-CG: Gauss-Newton right after
  // a Hessian solve that met negative curvature)
  int mode = prm->curvature;
  if (mode == HF_HYBRID) mode = *hybrid_state ? HF_GAUSS_NEWTON : HF_HESSIAN;

  // 3. the Newton system, from 0 or from eta delta_{k-1}
  const float* x0 = nullptr;
  if (prm->eta > 0.0f) {
    waxpy(Lc, x0v, nullptr, (double)prm->eta, delta, n);
    x0 = x0v;
  }
  const bool backtrack = prm->keep_cap > 0;
  const KeepPlan keep(prm->max_iters, prm->keep_cap, prm->keep_buf);
  rc = (prm->solver == HF_SOLVER_CG)
           ? solve_cg(c, W, Xc, yc, bc, g, prm->damping, prm->max_iters,
                      prm->rel_tol, mode, x0, s, d, &info->solve,
                      backtrack ? &keep : nullptr, minv)
           : solve_bicg(c, W, Xc, yc, bc, g, prm->damping, prm->max_iters,
                        prm->rel_tol, mode, x0, s, d, &info->solve,
                        backtrack ? &keep : nullptr, minv);
  if (rc != HF_OK) return rc;

  // objective at W + a v, reduced in fp64 (one full-batch forward)
  auto objective = [&](double a, const float* v, double* f) -> int {
    waxpy(Lc, wt, W, a, v, n);
    loss_only(c, wt, X, y, b, nullptr, scal + 4);
    HIP_TRY(c, hipMemcpyAsync(f, scal + 4, sizeof(double),
                              hipMemcpyDeviceToHost, c->stream));
    HIP_TRY(c, hipStreamSynchronize(c->stream));
    info->evals += 1;
    return HF_OK;
  };

  // CG-backtracking: from the final iterate back through the kept ones
  // (those formed before it) while f decreases
  const float* sb = s;          // the step candidate
  double f_sb = 0.0;
  info->backtrack_iter = -1;
  if (backtrack) {
    const int iters = info->solve.iters;
    int j_best = iters;
    if ((rc = objective(1.0, s, &f_sb))) return rc;
    for (int i = (int)keep.js.size() - 1; i >= 0; --i) {
      if (keep.js[i] >= iters) continue;
      const float* xj = keep.buf + (size_t)i * n;
      double fj;
      if ((rc = objective(1.0, xj, &fj))) return rc;
      if (!(fj < f_sb)) break;
      sb = xj;
      f_sb = fj;
      j_best = keep.js[i];
    }
    info->backtrack_iter = j_best;
    // the kept vectors sit n floats apart, so an earlier iterate may not be
    // 16-byte aligned: continue with an aligned copy (the warm start's
    // vector is free once the solve has run)
    if (sb != s) {
      waxpy(Lc, x0v, nullptr, 1.0, sb, n);
      sb = x0v;
    }
  }

  // 4. candidates: the step if it descends, and the oriented
  // negative-curvature direction rescaled to the solver's step length
  const float* da[4] = {g, s, g, d};
  const float* db[4] = {sb, s, d, d};
  dots4(Lc, da, db, n, c->Dp(c->oRed), scal);
  HIP_TRY(c, hipMemcpyAsync(hs, scal, 4 * sizeof(double), hipMemcpyDeviceToHost,
                            c->stream));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  const double gs = hs[0], ss = hs[1], gd = hs[2], dd = hs[3];
  const double gg = info->solve.rr0;
  struct Cand { int kind; const float* v; double scale, gTd; };
  Cand cand[2];
  int nc = 0;
  if (gs < 0.0) cand[nc++] = Cand{0, sb, 1.0, gs};
  if (info->solve.neg_curv && dd > 0.0) {
    const double target = ss > 0.0 ? std::sqrt(ss) : std::sqrt(gg);
    const double sc = target / std::sqrt(dd);
    cand[nc++] = Cand{1, d, sc, gd * sc};
  }

  // 5. Armijo backtracking for each candidate; keep the lower f
  int best = -1;
  double best_alpha = 0.0, best_f = f0;
  for (int k = 0; k < nc; ++k) {
    double alpha = 1.0;
    for (int t = 0; t <= prm->max_backtracks; ++t) {
      double ft;
      if (backtrack && cand[k].kind == 0 && t == 0) {
        ft = f_sb;                        // known from backtracking
      } else if ((rc = objective(alpha * cand[k].scale, cand[k].v, &ft))) {
        return rc;
      }
      if (ft <= f0 + (double)prm->armijo_c * alpha * cand[k].gTd) {
        if (best < 0 || ft < best_f) {
          best = k;
          best_alpha = alpha;
          best_f = ft;
        }
        break;
      }
      alpha *= (double)prm->shrink;
    }
  }

  // damping for the next iteration (Levenberg-Marquardt on rho); B p from a
  // stateless product at the old W (the line search has overwritten the
  // solve's activation cache)
  const double lam = (double)prm->damping;
  info->rho = std::nan("");
  info->damping_next = lam;
  if (prm->adapt_damping) {
    double rho = -INFINITY;
    if (best >= 0) {
      const Cand& cb = cand[best];
      float* q = c->F(c->oQ);
      if ((rc = hf_hvp(c, W, Xc, yc, Bc, cb.v, mode, q))) return rc;
      const float* ua[4] = {cb.v, cb.v, cb.v, cb.v};
      const float* ub[4] = {q, cb.v, q, cb.v};
      dots4(Lc, ua, ub, n, c->Dp(c->oRed), scal);
      HIP_TRY(c, hipMemcpyAsync(hs, scal, 2 * sizeof(double),
                                hipMemcpyDeviceToHost, c->stream));
      HIP_TRY(c, hipStreamSynchronize(c->stream));
      const double a = best_alpha * cb.scale;            // p = a v
      const double pBp = a * a * (hs[0] + lam * hs[1]);
      const double pred = best_alpha * cb.gTd + 0.5 * pBp;
      if (pred < 0.0) rho = (best_f - f0) / pred;
    }
    info->rho = rho;
    info->damping_next = rho < 0.25 ? 1.5 * lam : (rho > 0.75 ? lam * (2.0 / 3.0) : lam);
  }

  // 6. theta_{k+1} and delta_k
  info->mode_used = mode;
  info->f0 = f0;
  if (best >= 0) {
    const Cand& cb = cand[best];
    waxpy(Lc, W, W, best_alpha * cb.scale, cb.v, n);
    waxpy(Lc, delta, nullptr, cb.scale, cb.v, n);
    info->direction = cb.kind;
    info->accepted = 1;
    info->alpha = best_alpha;
    info->f1 = best_f;
    info->gTd = cb.gTd;
  } else {
    waxpy(Lc, delta, nullptr, 0.0, g, n);
    info->direction = -1;
    info->accepted = 0;
    info->alpha = 0.0;
    info->f1 = f0;
    info->gTd = 0.0;
  }
  if (prm->curvature == HF_HYBRID)
    *hybrid_state = (mode == HF_HESSIAN && info->solve.neg_curv) ? 1 : 0;
  HIP_TRY(c, hipGetLastError());
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  return HF_OK;
}

int hf_check(hf_ctx* c) {
  if (!c) return HF_EINVAL;
  if (!c->ws) return HF_OK;
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  int flag = 0;
  HIP_TRY(c, hipMemcpy(&flag, c->ws + c->oErr, sizeof(int), hipMemcpyDeviceToHost));
  if (flag) {
    int zero = 0;
    HIP_TRY(c, hipMemcpy(c->ws + c->oErr, &zero, sizeof(int), hipMemcpyHostToDevice));
    return fail(c, HF_ELABEL, "a label outside [0, %d) was seen", c->d[c->L]);
  }
  return HF_OK;
}

const char* hf_last_error(const hf_ctx* c) {
  if (!c) return "null context";
  return c->err.c_str();
}

const char* hf_build_id(void) { return HF_BUILD_ID; }

int hf_set_trace(hf_ctx* c, float* buf, int32_t cap) {
  if (!c) return HF_EINVAL;
  if (cap < 0) return fail(c, HF_EINVAL, "trace capacity %d < 0", cap);
  if (cap > 0 && !buf) return fail(c, HF_EINVAL, "trace buffer is NULL");
  if (cap > 0 && !a16(buf)) return fail(c, HF_EINVAL, "trace buffer is not 16-byte aligned");
  c->trace_buf = cap > 0 ? buf : nullptr;
  c->trace_cap = cap > 0 ? cap : 0;
  return HF_OK;
}

const char* hf_strerror(int32_t code) {
  switch (code) {
    case HF_OK: return "HF_OK";
    case HF_EINVAL: return "HF_EINVAL";
    case HF_ENOMEM: return "HF_ENOMEM";
    case HF_EHIP: return "HF_EHIP";
    case HF_ELABEL: return "HF_ELABEL";
    case HF_ENUMERIC: return "HF_ENUMERIC";
    case HF_EWORKSPACE: return "HF_EWORKSPACE";
    default: return "HF_UNKNOWN";
  }
}

int hf_prof_enable(hf_ctx* c, int32_t on) {
  if (!c) return HF_EINVAL;
  if (on && !c->prof) c->prof = new (std::nothrow) Profiler();
  if (on && !c->prof) return HF_ENOMEM;
  if (!on && c->prof) {
    delete c->prof;
    c->prof = nullptr;
  }
  return HF_OK;
}

int hf_prof_only(hf_ctx* c, const char* name) {
  if (!c || !c->prof) return HF_EINVAL;
  c->prof->only = name ? name : "";
  return HF_OK;
}

int hf_prof_reset(hf_ctx* c) {
  if (!c) return HF_EINVAL;
  if (c->prof) {
    c->prof->collect();
    c->prof->recs.clear();
    c->prof->index.clear();
  }
  return HF_OK;
}

int32_t hf_prof_count(hf_ctx* c) {
  if (!c || !c->prof) return 0;
  c->prof->collect();
  return (int32_t)c->prof->recs.size();
}

int hf_prof_get(hf_ctx* c, int32_t i, const char** name, int64_t* launches,
                double* total_ms, double* flops, double* bytes) {
  if (!c || !c->prof) return HF_EINVAL;
  c->prof->collect();
  if (i < 0 || i >= (int32_t)c->prof->recs.size()) return HF_EINVAL;
  const ProfRec& r = c->prof->recs[i];
  if (name) *name = r.name.c_str();
  if (launches) *launches = r.launches;
  if (total_ms) *total_ms = r.ms;
  if (flops) *flops = r.flops;
  if (bytes) *bytes = r.bytes;
  return HF_OK;
}

}  // extern "C"
