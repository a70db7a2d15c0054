// api.hip -- the extern "C" entry points declared in include/gcn.h.
//
// Every entry point validates its arguments on the host, plans its workspace
// with the same code for the size query and the real call, and enqueues
// kernels from the other translation units.  Nothing here allocates device
// memory.
#include <cstring>
#include <string>

#include "internal.h"

namespace gcn {

namespace {
thread_local std::string g_err;
}

gcn_status fail(gcn_status s, const std::string& msg) {
  g_err = msg;
  return s;
}

gcn_status hip_fail(hipError_t e, const char* what) {
  g_err = std::string(what) + ": " + hipGetErrorString(e);
  return GCN_E_HIP;
}

namespace {

// Workspace protocol: NULL buffer -> report size; else check it is large enough.
gcn_status ws_protocol(void* d_ws, size_t* ws_bytes, size_t need, const char* who, bool* query) {
  if (!ws_bytes) return fail(GCN_E_INVALID, std::string(who) + ": ws_bytes is NULL");
  if (!d_ws) {
    *ws_bytes = need;
    *query = true;
    return GCN_OK;
  }
  *query = false;
  if (*ws_bytes < need)
    return fail(GCN_E_CAPACITY, std::string(who) + ": workspace of " + std::to_string(*ws_bytes) +
                                    " bytes, " + std::to_string(need) + " needed");
  return GCN_OK;
}

gcn_status check_graph(const gcn_graph* g, const char* who) {
  if (!g) return fail(GCN_E_INVALID, std::string(who) + ": graph is NULL");
  if (g->n < 0) return fail(GCN_E_INVALID, std::string(who) + ": negative node count");
  if (g->n > 0 && (!g->row_ptr || !g->col_idx || !g->val))
    return fail(GCN_E_INVALID, std::string(who) + ": graph arrays missing");
  if (g->split.rows && g->split.n_long > 0 && (!g->split.first || !g->split.owner))
    return fail(GCN_E_INVALID, std::string(who) + ": split plan arrays missing");
  return GCN_OK;
}

gcn_status check_layer(const gcn_layer* L, const char* who) {
  if (!L) return fail(GCN_E_INVALID, std::string(who) + ": layer is NULL");
  if (L->f_in <= 0 || L->f_out <= 0) return fail(GCN_E_INVALID, std::string(who) + ": non-positive width");
  if (L->ld_in < L->f_in || L->ld_out < L->f_out)
    return fail(GCN_E_INVALID, std::string(who) + ": pitch smaller than width");
  if (L->act < GCN_ACT_NONE || L->act > GCN_ACT_SOFTMAX_CE)
    return fail(GCN_E_INVALID, std::string(who) + ": unknown activation");
  if (L->order < GCN_ORDER_AUTO || L->order > GCN_AGGREGATE_FIRST)
    return fail(GCN_E_INVALID, std::string(who) + ": unknown order");
  if (L->act == GCN_ACT_SOFTMAX_CE && L->f_out > 256)
    return fail(GCN_E_UNSUPPORTED, std::string(who) + ": softmax cross-entropy needs f_out <= 256");
  if (L->agg != GCN_AGG_NORM && L->agg != GCN_AGG_SUM && L->agg != GCN_AGG_MEAN && L->agg != GCN_AGG_MAX)
    return fail(GCN_E_INVALID, std::string(who) + ": unknown aggregator");
  if (L->agg == GCN_AGG_MAX && L->order == GCN_TRANSFORM_FIRST)
    return fail(GCN_E_INVALID, std::string(who) + ": a max layer aggregates first");
  if (L->agg == GCN_AGG_MAX && L->f_in > 256)
    return fail(GCN_E_UNSUPPORTED, std::string(who) + ": max aggregation needs f_in <= 256");
  return GCN_OK;
}

gcn_status check_sparse(const gcn_sparse_x* x, const gcn_graph* g, const gcn_layer* L, bool need_csc,
                        const char* who) {
  if (x->n != g->n || x->f != L->f_in)
    return fail(GCN_E_INVALID, std::string(who) + ": sparse X shape does not match graph / layer");
  if (!x->row_ptr || !x->col || !x->val) return fail(GCN_E_INVALID, std::string(who) + ": X_csr missing");
  if (need_csc && (!x->col_ptr || !x->row || !x->cval))
    return fail(GCN_E_INVALID, std::string(who) + ": X_csc missing");
  return GCN_OK;
}

int64_t pitch4(int64_t w) { return round_up(w, 4); }

// Pitch of a matrix whose rows are gathered (one random row per graph entry): the rows
// are fetched in 64-byte sectors, so of w rounded up to 4 or to 16 floats take the one
// whose rows touch fewer sectors on average over their offsets (41 floats: 3.5 sectors at
// pitch 44, 3 at pitch 48), the smaller on a tie.
double mean_sectors(int64_t w, int64_t pitch) {
  int64_t sum = 0;
  for (int64_t r = 0; r < 16; ++r) {
    const int64_t o = (4 * pitch * r) % 64;
    sum += (o + 4 * w + 63) / 64;
  }
  return (double)sum / 16.0;
}
int64_t gather_pitch(int64_t w) {
  const int64_t a = round_up(w, 4), b = round_up(w, 16);
  return mean_sectors(w, b) < mean_sectors(w, a) ? b : a;
}

int32_t resolve_order(const gcn_layer* L, bool x_sparse) {
  if (L->agg == GCN_AGG_MAX) return GCN_AGGREGATE_FIRST;  // max does not commute with W
  if (L->order != GCN_ORDER_AUTO) return L->order;
  if (L->act == GCN_ACT_SOFTMAX_CE || x_sparse) return GCN_TRANSFORM_FIRST;
  // aggregate-first aggregates f_in columns forward (and again backward above
  // layer 0); transform-first aggregates f_out columns in both passes
  const int64_t af = (int64_t)L->f_in * (L->index > 0 ? 2 : 1);
  return af < 2 * (int64_t)L->f_out ? GCN_AGGREGATE_FIRST : GCN_TRANSFORM_FIRST;
}

// The fused aggregate-first kernel serves 32 < f_in <= 128 in bf16x6 mode when
// GCN_AF_FUSED=1.  By default the layer runs as the aggregation followed by the
// row-panel GEMM, measured faster (arxiv-like layer 0: 229 + 100 us against 347 us;
// products-like 8.90 + 1.14 ms against 10.47 ms): the fused kernel's LDS and registers
// leave the gathers fewer wavefronts per CU than the standalone aggregation has.
bool af_fusable(int32_t f_in) {
  const char* e = getenv("GCN_AF_FUSED");
  if (!(e && e[0] == '1')) return false;
  return gemm_bf16x6_mode() && f_in > 32 && f_in <= 128;
}

// The aggregator that carries gradients back: A_hat and A + I are symmetric; the
// mean's transpose is (A + I) D^-1.
int32_t agg_transpose(int32_t agg) {
  if (agg == GCN_AGG_MEAN) return GCN_AGG_MEAN_T;
  if (agg == GCN_AGG_MEAN_T) return GCN_AGG_MEAN;
  return agg;
}

AggParams graph_agg(const gcn_graph* g, int32_t w, const float* M, int64_t ldm, float* Z, int64_t ldz,
                    int32_t agg = GCN_AGG_NORM) {
  AggParams p{};
  p.deg = g->deg;
  p.kind = agg == GCN_AGG_SUM ? AGG_W_ONE
           : agg == GCN_AGG_MEAN ? AGG_W_ROWMEAN
           : agg == GCN_AGG_MEAN_T ? AGG_W_COLMEAN : AGG_W_VAL;
  p.n = g->n;
  p.row_ptr = g->row_ptr;
  p.col = g->col_idx;
  p.val = g->val;
  p.M = M;
  p.ldm = ldm;
  p.w = w;
  p.Z = Z;
  p.ldz = ldz;
  p.epi = AGG_NONE;
  p.order = g->order;
  return p;
}

GemmParams gemm(int64_t m, int64_t n, int64_t k, const float* A, int64_t lda, bool ta, const float* B,
                int64_t ldb, bool tb, float* C, int64_t ldc) {
  GemmParams p{};
  p.m = m;
  p.n = n;
  p.k = k;
  p.A = A;
  p.lda = lda;
  p.ta = ta;
  p.B = B;
  p.ldb = ldb;
  p.tb = tb;
  p.C = C;
  p.ldc = ldc;
  p.epi = GEMM_NONE;
  return p;
}

// ---------------------------------------------------------------------------
// layer plans: the same function sizes the workspace (base == NULL) and runs
// ---------------------------------------------------------------------------

// relu_bits (optional, ReLU layers): also write the bitmask 1[H_out > 0] (relu_bits_words
// words per row) where the producing kernel can; *bits_written tells whether it does (set
// in the sizing pass too).
// The mean of the per-row losses; with db_out, the same fixed-order pass also sums the
// columns of G = dLoss/dZ (written to Hout by the loss epilogue), the layer's bias gradient,
// so that the backward pass need not read G again for it.
gcn_status loss_pass(int32_t n, const gcn_layer* L, const float* G, const float* row_loss, float* loss,
                     float* db_out, void* cws, hipStream_t s) {
  if (db_out) return launch_colsum(n, L->f_out, G, L->ld_out, db_out, row_loss, loss, cws, s);
  return launch_colsum(n, 0, nullptr, 0, nullptr, row_loss, loss, cws, s);
}

// X_csr W of a sparse first layer: lane slices of each row gather a row of W per entry
// (the aggregation kernel with the stored values of X).
gcn_status launch_spmm_xw(int64_t n, int64_t nnz, const int64_t* row_ptr, const int32_t* col, const float* val,
                          const float* W, int64_t ldw, int32_t w, float* C, int64_t ldc, hipStream_t s) {
  AggParams p{};
  p.n = (int32_t)n;
  p.row_ptr = row_ptr;
  p.col = col;
  p.val = val;
  p.M = W;
  p.ldm = ldw;
  p.w = w;
  p.Z = C;
  p.ldz = ldc;
  p.epi = AGG_NONE;
  p.tag = "spmm_xw";
  return launch_aggregate(p, nnz, nullptr, nullptr, s);
}

gcn_status layer_fwd(const gcn_graph* g, const gcn_layer* L, const float* Hin, const gcn_sparse_x* x,
                     const float* W, const float* b, float* Hout, float* saved, const int32_t* labels,
                     float* loss, float* logits, Arena& a, hipStream_t s, uint32_t* relu_bits = nullptr,
                     bool* bits_written = nullptr, float* db_out = nullptr, const SplitJob* sj = nullptr,
                     int nsj = 0) {
  const int32_t n = g->n;
  const int32_t order = resolve_order(L, x != nullptr);
  const bool run = a.base != nullptr;
  if (bits_written) *bits_written = false;
  const bool want_bits = relu_bits && L->act == GCN_ACT_RELU;
  if (order == GCN_AGGREGATE_FIRST) {
    // P = S H_in (kept for the backward pass), then H_out = act(P W + b): one fused
    // kernel when the widths allow it (bf16x6 mode, linear S), else an aggregation and a
    // GEMM.  The workspace covers both, so a size query made without buffers stays valid.
    // With the softmax cross-entropy, Z = P W + b goes through the loss epilogue of an
    // aggregation over the identity operator.
    const bool softmax = L->act == GCN_ACT_SOFTMAX_CE;
    const bool fusable = af_fusable(L->f_in) && L->agg != GCN_AGG_MAX && !softmax;
    size_t need = aggregate_workspace(&g->split, L->f_in);
    if (fusable) need = std::max(need, agg_gemm_workspace(&g->split, L->f_in, L->f_out));
    void* aws = a.take<char>((int64_t)need);
    const int64_t ldz = gather_pitch(L->f_out);
    float* Zs = softmax ? a.take<float>((int64_t)n * ldz) : nullptr;
    int64_t* id_ptr = softmax ? a.take<int64_t>((int64_t)n + 1) : nullptr;
    int32_t* id_col = softmax ? a.take<int32_t>(n) : nullptr;
    float* row_loss = softmax ? a.take<float>(n) : nullptr;
    void* cws = softmax ? a.take<char>((int64_t)colsum_workspace(n, L->f_out)) : nullptr;
    // H_out = P W (+ b) when the fused kernel does not run (split weight in the workspace)
    GemmParams q = gemm(n, L->f_out, L->f_in, saved, L->ld_in, false, W, L->f_out, false, softmax ? Zs : Hout,
                        softmax ? ldz : L->ld_out);
    q.bias = b;
    void* gws = a.take<char>((int64_t)gemm_workspace(q));
    if (run && L->agg == GCN_AGG_MAX) {
      AggParams p = graph_agg(g, L->f_in, Hin, L->ld_in, saved, L->ld_in);
      int32_t* arg = reinterpret_cast<int32_t*>(saved + (int64_t)n * L->ld_in);
      GCN_TRY(launch_aggregate_max(p, g->nnz, saved, L->ld_in, arg, L->ld_in, s));
    }
    if (run && softmax) {
      if (L->agg != GCN_AGG_MAX) {
        AggParams p = graph_agg(g, L->f_in, Hin, L->ld_in, saved, L->ld_in, L->agg);
        GCN_TRY(launch_aggregate(p, g->nnz, &g->split, aws, s));
      }
      GCN_TRY(launch_gemm(with_split(q, sj, nsj), gws, s));
      GCN_TRY(launch_identity_csr(n, id_ptr, id_col, s));
      AggParams z{};
      z.n = n;
      z.row_ptr = id_ptr;
      z.col = id_col;
      z.kind = AGG_W_ONE;
      z.M = Zs;
      z.ldm = ldz;
      z.w = L->f_out;
      z.Z = Hout;
      z.ldz = L->ld_out;
      z.epi = AGG_SOFTMAX;
      z.labels = labels;
      z.row_loss = row_loss;
      z.logits = logits;
      z.ldl = L->ld_out;
      z.inv_n = n > 0 ? 1.f / (float)n : 0.f;
      z.tag = "softmax_ce";
      GCN_TRY(launch_aggregate(z, n, nullptr, nullptr, s));
      GCN_TRY(loss_pass(n, L, Hout, row_loss, loss, db_out, cws, s));
      return GCN_OK;
    }
    q.epi = L->act == GCN_ACT_RELU ? GEMM_RELU : GEMM_NONE;
    const bool fused = fusable && agg_gemm_supported(L->f_in, L->ld_in, L->ld_in, Hin, saved);
    if (want_bits && !fused && gemm_rows_supported(q)) {
      q.relu_bits = relu_bits;
      q.ld_relu_bits = relu_bits_words(L->f_out);
      if (bits_written) *bits_written = true;
    }
    if (run && L->agg == GCN_AGG_MAX) {
      GCN_TRY(launch_gemm(with_split(q, sj, nsj), gws, s));
      return GCN_OK;
    }
    if (run) {
      AggParams p = graph_agg(g, L->f_in, Hin, L->ld_in, saved, L->ld_in, L->agg);
      if (fused) {
        GCN_TRY(launch_agg_gemm(p, g->nnz, &g->split, W, L->f_out, L->f_out, b, L->act == GCN_ACT_RELU, Hout,
                                L->ld_out, aws, s));
      } else {
        GCN_TRY(launch_aggregate(p, g->nnz, &g->split, aws, s));
        GCN_TRY(launch_gemm(with_split(q, sj, nsj), gws, s));
      }
    }
    return GCN_OK;
  }
  // transform-first: M = H_in W (or X_csr W), then Z = A_hat M + b with the epilogue
  const int64_t ldm = gather_pitch(L->f_out);
  float* M = a.take<float>((int64_t)n * ldm);
  float* row_loss = L->act == GCN_ACT_SOFTMAX_CE ? a.take<float>(n) : nullptr;
  void* cws = L->act == GCN_ACT_SOFTMAX_CE ? a.take<char>((int64_t)colsum_workspace(n, L->f_out)) : nullptr;
  void* aws = a.take<char>((int64_t)aggregate_workspace(&g->split, L->f_out));
  const GemmParams q = gemm(n, L->f_out, L->f_in, Hin, L->ld_in, false, W, L->f_out, false, M, ldm);
  void* gws = x ? nullptr : a.take<char>((int64_t)gemm_workspace(q));
  if (bits_written) *bits_written = want_bits;  // the aggregation epilogue writes them
  if (!run) return GCN_OK;
  if (x) {
    GCN_TRY(launch_spmm_xw(n, x->nnz, x->row_ptr, x->col, x->val, W, L->f_out, L->f_out, M, ldm, s));
  } else {
    GCN_TRY(launch_gemm(with_split(q, sj, nsj), gws, s));
  }
  AggParams p = graph_agg(g, L->f_out, M, ldm, Hout, L->ld_out, L->agg);
  p.bias = b;
  if (L->act == GCN_ACT_RELU) p.epi = AGG_RELU;
  if (want_bits) {
    p.relu_bits = relu_bits;
    p.ld_relu_bits = relu_bits_words(L->f_out);
  }
  if (L->act == GCN_ACT_SOFTMAX_CE) {
    p.epi = AGG_SOFTMAX;
    p.labels = labels;
    p.row_loss = row_loss;
    p.logits = logits;
    p.ldl = L->ld_out;
    p.inv_n = n > 0 ? 1.f / (float)n : 0.f;
  }
  GCN_TRY(launch_aggregate(p, g->nnz, &g->split, aws, s));
  if (L->act == GCN_ACT_SOFTMAX_CE) GCN_TRY(loss_pass(n, L, Hout, row_loss, loss, db_out, cws, s));
  return GCN_OK;
}

// mask_bits (optional): the bitmask 1[H_in > 0] written by the previous layer's forward;
// the transform-first input gradient reads it instead of H_in where the row-panel product
// serves it; *bits_used tells whether it does (set in the sizing pass too).  On that path
// the product also writes the column sums of G_prev into db_prev when given (the bias
// gradient of the layer below; *db_prev_done).  db_ready: db was written that way already.
gcn_status layer_bwd(const gcn_graph* g, const gcn_layer* L, const float* G, const float* Hin,
                     const gcn_sparse_x* x, const float* saved, const float* W, float* dW, float* db,
                     float* Gprev, Arena& a, hipStream_t s, const uint32_t* mask_bits = nullptr,
                     bool* bits_used = nullptr, float* db_prev = nullptr, bool* db_prev_done = nullptr,
                     bool db_ready = false, const SplitJob* sj = nullptr, int nsj = 0) {
  const int32_t n = g->n;
  const int32_t order = resolve_order(L, x != nullptr);
  const bool run = a.base != nullptr;
  if (bits_used) *bits_used = false;
  if (db_prev_done) *db_prev_done = false;
  void* cws = a.take<char>((int64_t)colsum_workspace(n, L->f_out));
  if (order == GCN_AGGREGATE_FIRST) {
    // Z = P W + b with P = A_hat H_in: dW = P^T G; dP = G W^T; G_prev = (A_hat dP) * 1[H_in > 0]
    GemmParams dw = gemm(L->f_in, L->f_out, n, saved, L->ld_in, true, G, L->ld_out, false, dW, L->f_out);
    void* gws = a.take<char>((int64_t)gemm_workspace(dw));
    const int64_t ldt = gather_pitch(L->f_in);
    float* T = Gprev ? a.take<float>((int64_t)n * ldt) : nullptr;
    void* aws = Gprev ? a.take<char>((int64_t)aggregate_workspace(&g->split, L->f_in)) : nullptr;
    const GemmParams t = gemm(n, L->f_in, L->f_out, G, L->ld_out, false, W, L->f_out, true, T, ldt);
    void* tws = Gprev ? a.take<char>((int64_t)gemm_workspace(t)) : nullptr;
    if (!run) return GCN_OK;
    GCN_TRY(launch_gemm(dw, gws, s));
    if (!db_ready) GCN_TRY(launch_colsum(n, L->f_out, G, L->ld_out, db, nullptr, nullptr, cws, s));
    if (Gprev) {
      GCN_TRY(launch_gemm(with_split(t, sj, nsj), tws, s));
      AggParams p = graph_agg(g, L->f_in, T, ldt, Gprev, L->ld_in, agg_transpose(L->agg));
      if (L->agg == GCN_AGG_MAX) {
        // each (G W^T)[v,c] goes back to the saved maximiser of (v, c)
        const int32_t* arg = reinterpret_cast<const int32_t*>(saved + (int64_t)n * L->ld_in);
        GCN_TRY(launch_aggregate_max_bwd(p, g->nnz, arg, L->ld_in, Hin, L->ld_in, Gprev, L->ld_in, s));
        return GCN_OK;
      }
      p.epi = AGG_MASK;
      p.mask = Hin;
      p.ldmask = L->ld_in;
      GCN_TRY(launch_aggregate(p, g->nnz, &g->split, aws, s));
    }
    return GCN_OK;
  }
  // transform-first: Q = S^T G; dW = H_in^T Q (X_csc Q); G_prev = (Q W^T) * 1[H_in > 0]
  const int64_t ldq = pitch4(L->f_out);
  float* Q = a.take<float>((int64_t)n * ldq);
  GemmParams dw = gemm(L->f_in, L->f_out, n, Hin, L->ld_in, true, Q, ldq, false, dW, L->f_out);
  void* gws = x ? nullptr : a.take<char>((int64_t)gemm_workspace(dw));
  const size_t agg_need = std::max(aggregate_workspace(&g->split, L->f_out),
                                   x && x->col_ptr ? spmm_xt_workspace(n, x->f, x->nnz, L->f_out, &x->csc_split)
                                                   : (size_t)0);
  void* aws = a.take<char>((int64_t)agg_need);
  GemmParams t = gemm(n, L->f_in, L->f_out, Q, ldq, false, W, L->f_out, true, Gprev, L->ld_in);
  t.epi = GEMM_MASK;
  t.mask = Hin;
  t.ldmask = L->ld_in;
  if (mask_bits && Gprev) {
    GemmParams tb = t;
    tb.mask_bits = mask_bits;
    tb.ld_mask_bits = relu_bits_words(L->f_in);
    if (gemm_rows_supported(tb)) {
      t = tb;
      if (bits_used) *bits_used = true;
      if (db_prev) {
        t.colsum = db_prev;
        if (db_prev_done) *db_prev_done = true;
      }
    }
  }
  void* tws = Gprev ? a.take<char>((int64_t)gemm_workspace(t)) : nullptr;
  if (!run) return GCN_OK;
  GCN_TRY(launch_aggregate(graph_agg(g, L->f_out, G, L->ld_out, Q, ldq, agg_transpose(L->agg)), g->nnz,
                           &g->split, aws, s));
  if (x && !x->col_ptr) {
    // no CSC view: dW = X^T Q by atomic adds from the CSR rows (Section IV-D)
    GCN_TRY(launch_spmm_t_atomic(n, x->row_ptr, x->col, x->val, Q, ldq, L->f_out, x->f, dW, L->f_out, x->nnz, s));
  } else if (x) {
    // dW = X^T Q from the CSC view (tiled by row chunks where that pays)
    GCN_TRY(launch_spmm_xt(n, x->f, x->nnz, x->col_ptr, x->row, x->cval, &x->csc_split, Q, ldq, L->f_out, dW,
                           L->f_out, aws, s));
  } else {
    GCN_TRY(launch_gemm(dw, gws, s));
  }
  if (!db_ready) GCN_TRY(launch_colsum(n, L->f_out, G, L->ld_out, db, nullptr, nullptr, cws, s));
  if (Gprev) GCN_TRY(launch_gemm(with_split(t, sj, nsj), tws, s));
  return GCN_OK;
}

gcn_status validate_fwd(const gcn_graph* g, const gcn_layer* L, const float* Hin, const gcn_sparse_x* x,
                        const float* W, float* Hout, float* saved, const int32_t* labels, float* loss,
                        const char* who) {
  GCN_TRY(check_graph(g, who));
  GCN_TRY(check_layer(L, who));
  if ((Hin == nullptr) == (x == nullptr))
    return fail(GCN_E_INVALID, std::string(who) + ": exactly one of d_Hin and x must be given");
  if (x) GCN_TRY(check_sparse(x, g, L, false, who));
  if (!W || !Hout) return fail(GCN_E_INVALID, std::string(who) + ": d_W and d_Hout are required");
  const int32_t order = resolve_order(L, x != nullptr);
  if (order == GCN_AGGREGATE_FIRST) {
    if (x) return fail(GCN_E_UNSUPPORTED, std::string(who) + ": aggregate-first needs dense input");
    if (!saved) return fail(GCN_E_INVALID, std::string(who) + ": aggregate-first needs d_saved");
  }
  if (L->act == GCN_ACT_SOFTMAX_CE && (!labels || !loss))
    return fail(GCN_E_INVALID, std::string(who) + ": softmax cross-entropy needs labels and d_loss");
  return GCN_OK;
}

gcn_status validate_bwd(const gcn_graph* g, const gcn_layer* L, const float* G, const float* Hin,
                        const gcn_sparse_x* x, const float* saved, const float* W, float* dW, float* db,
                        float* Gprev, const char* who) {
  GCN_TRY(check_graph(g, who));
  GCN_TRY(check_layer(L, who));
  if (!G || !W || !dW || !db) return fail(GCN_E_INVALID, std::string(who) + ": G, W, dW and db are required");
  if (x) {
    GCN_TRY(check_sparse(x, g, L, false, who));  // without X_csc: the atomic implicit transpose
    if (!x->col_ptr && L->f_out > 256)
      return fail(GCN_E_UNSUPPORTED, std::string(who) + ": the atomic transpose product needs f_out <= 256");
    if (Gprev) return fail(GCN_E_INVALID, std::string(who) + ": no input gradient for sparse X");
  } else if (!Hin) {
    return fail(GCN_E_INVALID, std::string(who) + ": d_Hin is required for a dense input");
  }
  const int32_t order = resolve_order(L, x != nullptr);
  if (order == GCN_AGGREGATE_FIRST && !saved)
    return fail(GCN_E_INVALID, std::string(who) + ": aggregate-first needs d_saved");
  if (order == GCN_AGGREGATE_FIRST && x)
    return fail(GCN_E_UNSUPPORTED, std::string(who) + ": aggregate-first needs dense input");
  return GCN_OK;
}

}  // namespace
}  // namespace gcn

using namespace gcn;

extern "C" {

const char* gcn_status_string(gcn_status s) {
  switch (s) {
    case GCN_OK: return "GCN_OK";
    case GCN_E_INVALID: return "GCN_E_INVALID";
    case GCN_E_RANGE: return "GCN_E_RANGE";
    case GCN_E_OVERFLOW: return "GCN_E_OVERFLOW";
    case GCN_E_CAPACITY: return "GCN_E_CAPACITY";
    case GCN_E_HIP: return "GCN_E_HIP";
    case GCN_E_UNSUPPORTED: return "GCN_E_UNSUPPORTED";
    default: return "GCN_E_UNKNOWN";
  }
}

const char* gcn_last_error(void) { return g_err.c_str(); }

int32_t gcn_version(void) { return 3; }

int32_t gcn_layer_order(const gcn_layer* L, int32_t x_sparse) {
  return L ? resolve_order(L, x_sparse != 0) : GCN_TRANSFORM_FIRST;
}

gcn_status gcn_build_csr(int32_t n, int64_t n_edges, const int32_t* d_src, const int32_t* d_dst,
                         gcn_graph* g, void* d_ws, size_t* ws_bytes, hipStream_t stream) {
  g_err.clear();
  if (n < 0 || n_edges < 0) return fail(GCN_E_INVALID, "gcn_build_csr: negative size");
  if (n_edges >= (int64_t(1) << 30))
    return fail(GCN_E_OVERFLOW, "gcn_build_csr: more than 2^30 input pairs (row counts are int32)");
  bool query = false;
  GCN_TRY(ws_protocol(d_ws, ws_bytes, build_csr_workspace(n, n_edges), "gcn_build_csr", &query));
  if (query) return GCN_OK;
  if (!g) return fail(GCN_E_INVALID, "gcn_build_csr: graph is NULL");
  if (n_edges > 0 && (!d_src || !d_dst)) return fail(GCN_E_INVALID, "gcn_build_csr: edge arrays missing");
  if (!g->row_ptr || (n > 0 && (!g->deg || !g->dinv || !g->col_idx || !g->val)))
    return fail(GCN_E_INVALID, "gcn_build_csr: output arrays missing");
  if (g->split.rows && (!g->split.first || !g->split.owner || g->split.cap < 0))
    return fail(GCN_E_INVALID, "gcn_build_csr: split plan arrays missing");
  if (g->nnz_cap < 0) return fail(GCN_E_INVALID, "gcn_build_csr: negative capacity");
  g->n = n;
  return run_build_csr(n, n_edges, d_src, d_dst, g, d_ws, stream);
}

gcn_status gcn_feature_stats(const float* d_X, int32_t n, int32_t f, int64_t ldx, int32_t tau_num,
                             int32_t tau_den, int32_t force_mode, int64_t* d_row_nnz,
                             gcn_feature_info* info, gcn_sparse_x* x, void* d_ws, size_t* ws_bytes,
                             hipStream_t stream) {
  g_err.clear();
  if (n < 0 || f < 0 || ldx < f) return fail(GCN_E_INVALID, "gcn_feature_stats: bad shape or pitch");
  if (tau_den <= 0 || tau_num < 0) return fail(GCN_E_INVALID, "gcn_feature_stats: tau must be >= 0 with tau_den > 0");
  if (force_mode < -1 || force_mode > GCN_SPARSE) return fail(GCN_E_INVALID, "gcn_feature_stats: bad force_mode");
  const bool csc = x && x->col_ptr;
  bool query = false;
  GCN_TRY(ws_protocol(d_ws, ws_bytes, feature_stats_workspace(n, f, csc), "gcn_feature_stats", &query));
  if (query) return GCN_OK;
  if (!info || (n > 0 && f > 0 && !d_X)) return fail(GCN_E_INVALID, "gcn_feature_stats: X and info are required");
  if (x && (!x->row_ptr || !x->col || !x->val || (csc && (!x->row || !x->cval))))
    return fail(GCN_E_INVALID, "gcn_feature_stats: sparse output arrays missing");
  if (x && csc && x->csc_split.rows && (!x->csc_split.first || !x->csc_split.owner || x->csc_split.cap < 0))
    return fail(GCN_E_INVALID, "gcn_feature_stats: split plan arrays missing");
  return run_feature_stats(d_X, n, f, ldx, tau_num, tau_den, force_mode, d_row_nnz, info, x, d_ws, stream);
}

gcn_status gcn_layer_fwd(const gcn_graph* g, const gcn_layer* L, const float* d_Hin,
                         const gcn_sparse_x* x, const float* d_W, const float* d_b, float* d_Hout,
                         float* d_saved, const int32_t* d_labels, float* d_loss, float* d_logits,
                         void* d_ws, size_t* ws_bytes, hipStream_t stream) {
  g_err.clear();
  GCN_TRY(validate_fwd(g, L, d_Hin, x, d_W, d_Hout, d_saved, d_labels, d_loss, "gcn_layer_fwd"));
  Arena plan;
  GCN_TRY(layer_fwd(g, L, d_Hin, x, d_W, d_b, d_Hout, d_saved, d_labels, d_loss, d_logits, plan, stream));
  bool query = false;
  GCN_TRY(ws_protocol(d_ws, ws_bytes, plan.used, "gcn_layer_fwd", &query));
  if (query) return GCN_OK;
  Arena a;
  a.base = static_cast<char*>(d_ws);
  return layer_fwd(g, L, d_Hin, x, d_W, d_b, d_Hout, d_saved, d_labels, d_loss, d_logits, a, stream);
}

gcn_status gcn_layer_bwd(const gcn_graph* g, const gcn_layer* L, const float* d_G, const float* d_Hin,
                         const gcn_sparse_x* x, const float* d_saved, const float* d_W, float* d_dW,
                         float* d_db, float* d_Gprev, void* d_ws, size_t* ws_bytes, hipStream_t stream) {
  g_err.clear();
  GCN_TRY(validate_bwd(g, L, d_G, d_Hin, x, d_saved, d_W, d_dW, d_db, d_Gprev, "gcn_layer_bwd"));
  Arena plan;
  GCN_TRY(layer_bwd(g, L, d_G, d_Hin, x, d_saved, d_W, d_dW, d_db, d_Gprev, plan, stream));
  bool query = false;
  GCN_TRY(ws_protocol(d_ws, ws_bytes, plan.used, "gcn_layer_bwd", &query));
  if (query) return GCN_OK;
  Arena a;
  a.base = static_cast<char*>(d_ws);
  return layer_bwd(g, L, d_G, d_Hin, x, d_saved, d_W, d_dW, d_db, d_Gprev, a, stream);
}

gcn_status gcn_epoch(gcn_model* m, const gcn_graph* g, const float* d_X, const gcn_sparse_x* x,
                     const int32_t* d_labels, float* d_loss, void* d_ws, size_t* ws_bytes,
                     hipStream_t stream) {
  g_err.clear();
  const char* who = "gcn_epoch";
  if (!m || !m->layers || m->n_layers <= 0) return fail(GCN_E_INVALID, "gcn_epoch: model has no layers");
  const int L = m->n_layers;
  if (2 * L > 16) return fail(GCN_E_UNSUPPORTED, "gcn_epoch: at most 8 layers");
  if (!m->W || !m->b || !m->dW || !m->db || !m->mW || !m->vW || !m->mb || !m->vb || !m->act || !m->grad)
    return fail(GCN_E_INVALID, "gcn_epoch: model pointer arrays missing");
  for (int l = 0; l < L; ++l) {
    const gcn_layer* ly = &m->layers[l];
    GCN_TRY(check_layer(ly, who));
    if (ly->index != l) return fail(GCN_E_INVALID, "gcn_epoch: layers[l].index must be l");
    if (l > 0 && (ly->f_in != m->layers[l - 1].f_out || ly->ld_in != m->layers[l - 1].ld_out))
      return fail(GCN_E_INVALID, "gcn_epoch: consecutive layer widths / pitches disagree");
    if ((l == L - 1) != (ly->act == GCN_ACT_SOFTMAX_CE))
      return fail(GCN_E_INVALID, "gcn_epoch: softmax cross-entropy must be the last layer's activation");
    // the backward of layer l + 1 multiplies by 1[H_{l+1} > 0], the derivative of ReLU,
    // so a hidden layer without it would get wrong gradients
    if (l < L - 1 && ly->act != GCN_ACT_RELU)
      return fail(GCN_E_UNSUPPORTED, "gcn_epoch: every hidden layer's activation must be ReLU");
    if (!m->W[l] || !m->dW[l] || !m->db[l] || !m->mW[l] || !m->vW[l] || !m->grad[l] || !m->b[l] ||
        !m->mb[l] || !m->vb[l] || (l < L - 1 && !m->act[l]))
      return fail(GCN_E_INVALID, "gcn_epoch: a layer buffer is NULL");
  }
  // Validate every layer call, then plan the workspace: a prefix holding the ReLU
  // bitmasks that live from a layer's forward to the next layer's backward (kept where the
  // producing epilogue can write them and that backward can read them), then the maximum
  // over the layer calls.  The sizing pass runs with a stand-in address for the bits.
  uint32_t* const probe = reinterpret_cast<uint32_t*>((uintptr_t)256);
  float* const probe_db = reinterpret_cast<float*>((uintptr_t)256);
  bool writes[8] = {}, reads[8] = {}, sums[8] = {};  // sums[l]: layer l's backward can write db[l-1]
  size_t need = 0;
  for (int l = 0; l < L; ++l) {
    const gcn_layer* ly = &m->layers[l];
    const float* Hin = l == 0 ? d_X : m->act[l - 1];
    const gcn_sparse_x* xl = l == 0 ? x : nullptr;
    float* Hout = l < L - 1 ? m->act[l] : m->grad[l];
    float* saved = m->saved ? m->saved[l] : nullptr;
    GCN_TRY(validate_fwd(g, ly, Hin, xl, m->W[l], Hout, saved, d_labels, d_loss, who));
    GCN_TRY(validate_bwd(g, ly, m->grad[l], Hin, xl, saved, m->W[l], m->dW[l], m->db[l],
                         l > 0 ? m->grad[l - 1] : nullptr, who));
    Arena pf, pb;
    GCN_TRY(layer_fwd(g, ly, Hin, xl, m->W[l], m->b[l], Hout, saved, d_labels, d_loss, nullptr, pf, stream,
                      l < L - 1 ? probe : nullptr, &writes[l]));
    GCN_TRY(layer_bwd(g, ly, m->grad[l], Hin, xl, saved, m->W[l], m->dW[l], m->db[l],
                      l > 0 ? m->grad[l - 1] : nullptr, pb, stream, l > 0 ? probe : nullptr, &reads[l],
                      l > 0 ? probe_db : nullptr, &sums[l]));
    need = std::max(need, std::max(pf.used, pb.used));
  }
  int64_t bits_at[8];
  size_t bits_bytes = 0;
  for (int l = 0; l < L; ++l) {
    bits_at[l] = -1;
    if (l < L - 1 && writes[l] && reads[l + 1]) {
      bits_at[l] = (int64_t)bits_bytes;
      bits_bytes += (size_t)round_up((int64_t)g->n * relu_bits_words(m->layers[l].f_out) * 4, 256);
    }
  }
  // Every weight in the two forms the row-panel products take it in (W for H W, W^T for
  // the input gradient), split once at the start: the weights change only in the Adam
  // step at the end.  A product that does not take the row-panel kernel ignores its job.
  // GCN_EPOCH_PREP=0 turns both epoch-level shortcuts off (this split and the bias
  // gradient of the loss pass): the products then split their own weights and the
  // backward pass sums G itself, with bitwise the same results.
  const char* prep_env = getenv("GCN_EPOCH_PREP");
  const bool prep = !(prep_env && strcmp(prep_env, "0") == 0);
  SplitJob jobs[kMaxSplitJobs];
  int njobs = 0;
  int64_t job_at[kMaxSplitJobs];
  for (int l = 0; l < L && prep; ++l) {
    const int64_t fi = m->layers[l].f_in, fo = m->layers[l].f_out;
    const float* const aligned_probe = reinterpret_cast<const float*>((uintptr_t)256);
    for (int form = 0; form < 2; ++form) {
      const bool tb = form == 1;
      if (tb && l == 0) continue;           // no input gradient below layer 0
      if (!tb && l == 0 && x) continue;     // sparse X: the first product is X_csr W
      const int64_t k = tb ? fo : fi, n = tb ? fi : fo;
      const GemmParams probe = gemm(g->n, n, k, aligned_probe, round_up(k, 4), false, m->W[l], fo, tb, nullptr, n);
      if (!gemm_rows_supported(probe) || njobs == kMaxSplitJobs) continue;
      jobs[njobs] = SplitJob{m->W[l], fo, tb, k, n, nullptr};
      job_at[njobs] = (int64_t)bits_bytes;
      bits_bytes += gemm_rows_split_bytes(jobs[njobs]);
      ++njobs;
    }
  }
  bool query = false;
  GCN_TRY(ws_protocol(d_ws, ws_bytes, bits_bytes + need, who, &query));
  if (query) return GCN_OK;
  char* const base = static_cast<char*>(d_ws);
  auto bits_of = [&](int l) { return bits_at[l] < 0 ? nullptr : reinterpret_cast<uint32_t*>(base + bits_at[l]); };
  for (int q = 0; q < njobs; ++q) jobs[q].out = base + job_at[q];
  GCN_TRY(launch_split_batch(jobs, njobs, stream));
  for (int l = 0; l < L; ++l) {
    Arena a;
    a.base = base + bits_bytes;
    const gcn_layer* ly = &m->layers[l];
    GCN_TRY(layer_fwd(g, ly, l == 0 ? d_X : m->act[l - 1], l == 0 ? x : nullptr, m->W[l], m->b[l],
                      l < L - 1 ? m->act[l] : m->grad[l], m->saved ? m->saved[l] : nullptr, d_labels,
                      d_loss, nullptr, a, stream, bits_of(l), nullptr, prep && l == L - 1 ? m->db[l] : nullptr,
                      jobs, njobs));
  }
  // with the bitmask, layer l's input-gradient product also sums the columns of G_{l-1}
  // (db of layer l - 1), which then skips its own column-sum pass over G_{l-1}; the last
  // layer's bias gradient comes out of the loss pass of the forward
  bool db_from_above[8] = {};
  db_from_above[L - 1] = prep;
  for (int l = L - 1; l >= 0; --l) {
    Arena a;
    a.base = base + bits_bytes;
    const gcn_layer* ly = &m->layers[l];
    const bool fuse_db = l > 0 && bits_at[l - 1] >= 0 && sums[l];
    GCN_TRY(layer_bwd(g, ly, m->grad[l], l == 0 ? d_X : m->act[l - 1], l == 0 ? x : nullptr,
                      m->saved ? m->saved[l] : nullptr, m->W[l], m->dW[l], m->db[l],
                      l > 0 ? m->grad[l - 1] : nullptr, a, stream, l > 0 ? bits_of(l - 1) : nullptr, nullptr,
                      fuse_db ? m->db[l - 1] : nullptr, nullptr, db_from_above[l], jobs, njobs));
    if (fuse_db) db_from_above[l - 1] = true;
  }
  gcn_adam_tensor t[16];
  for (int l = 0; l < L; ++l) {
    const int64_t fi = m->layers[l].f_in, fo = m->layers[l].f_out;
    t[2 * l] = gcn_adam_tensor{m->W[l], m->dW[l], m->mW[l], m->vW[l], fi * fo};
    t[2 * l + 1] = gcn_adam_tensor{m->b[l], m->db[l], m->mb[l], m->vb[l], fo};
  }
  GCN_TRY(launch_adam(t, 2 * L, m->step + 1, m->d_step, m->lr, m->beta1, m->beta2, m->eps, stream));
  if (!m->d_step) m->step += 1;
  return GCN_OK;
}

gcn_status gcn_aggregate(const gcn_graph* g, int32_t agg, int32_t w, const float* d_M, int64_t ldm,
                         const float* d_bias, int32_t epi, const float* d_mask, int64_t ldmask, float* d_Z,
                         int64_t ldz, void* d_ws, size_t* ws_bytes, hipStream_t stream) {
  g_err.clear();
  GCN_TRY(check_graph(g, "gcn_aggregate"));
  if (agg < GCN_AGG_NORM || agg > GCN_AGG_MEAN_T)
    return fail(GCN_E_INVALID, "gcn_aggregate: aggregator must be NORM, SUM, MEAN or MEAN_T");
  if (w < 0 || ldm < w || ldz < w) return fail(GCN_E_INVALID, "gcn_aggregate: bad width or pitch");
  if (epi < GCN_EPI_NONE || epi > GCN_EPI_MASK) return fail(GCN_E_INVALID, "gcn_aggregate: unknown epilogue");
  if (epi == GCN_EPI_MASK && (!d_mask || ldmask < w)) return fail(GCN_E_INVALID, "gcn_aggregate: mask missing");
  bool query = false;
  GCN_TRY(ws_protocol(d_ws, ws_bytes, aggregate_workspace(&g->split, w), "gcn_aggregate", &query));
  if (query) return GCN_OK;
  if (g->n > 0 && w > 0 && (!d_M || !d_Z)) return fail(GCN_E_INVALID, "gcn_aggregate: d_M and d_Z are required");
  AggParams p = graph_agg(g, w, d_M, ldm, d_Z, ldz, agg);
  p.bias = d_bias;
  p.epi = epi == GCN_EPI_RELU ? AGG_RELU : (epi == GCN_EPI_MASK ? AGG_MASK : AGG_NONE);
  p.mask = d_mask;
  p.ldmask = ldmask;
  return launch_aggregate(p, g->nnz, &g->split, d_ws, stream);
}

gcn_status gcn_aggregate_max(const gcn_graph* g, int32_t w, const float* d_M, int64_t ldm, float* d_P,
                             int64_t ldp, int32_t* d_arg, int64_t ldarg, void* d_ws, size_t* ws_bytes,
                             hipStream_t stream) {
  g_err.clear();
  GCN_TRY(check_graph(g, "gcn_aggregate_max"));
  if (w < 0 || ldm < w || ldp < w || ldarg < w) return fail(GCN_E_INVALID, "gcn_aggregate_max: bad width or pitch");
  if (w > 256) return fail(GCN_E_UNSUPPORTED, "gcn_aggregate_max: width above 256");
  bool query = false;
  GCN_TRY(ws_protocol(d_ws, ws_bytes, 0, "gcn_aggregate_max", &query));
  if (query) return GCN_OK;
  if (g->n > 0 && w > 0 && (!d_M || !d_P || !d_arg)) return fail(GCN_E_INVALID, "gcn_aggregate_max: NULL buffer");
  return launch_aggregate_max(graph_agg(g, w, d_M, ldm, d_P, ldp), g->nnz, d_P, ldp, d_arg, ldarg, stream);
}

gcn_status gcn_aggregate_max_bwd(const gcn_graph* g, int32_t w, const float* d_dP, int64_t ldd,
                                 const int32_t* d_arg, int64_t ldarg, const float* d_mask, int64_t ldmask,
                                 float* d_dM, int64_t ldo, void* d_ws, size_t* ws_bytes, hipStream_t stream) {
  g_err.clear();
  GCN_TRY(check_graph(g, "gcn_aggregate_max_bwd"));
  if (w < 0 || ldd < w || ldarg < w || ldo < w || (d_mask && ldmask < w))
    return fail(GCN_E_INVALID, "gcn_aggregate_max_bwd: bad width or pitch");
  if (w > 256) return fail(GCN_E_UNSUPPORTED, "gcn_aggregate_max_bwd: width above 256");
  bool query = false;
  GCN_TRY(ws_protocol(d_ws, ws_bytes, 0, "gcn_aggregate_max_bwd", &query));
  if (query) return GCN_OK;
  if (g->n > 0 && w > 0 && (!d_dP || !d_arg || !d_dM))
    return fail(GCN_E_INVALID, "gcn_aggregate_max_bwd: NULL buffer");
  return launch_aggregate_max_bwd(graph_agg(g, w, d_dP, ldd, d_dM, ldo), g->nnz, d_arg, ldarg, d_mask, ldmask,
                                  d_dM, ldo, stream);
}

gcn_status gcn_gemm(int32_t op, int64_t m, int64_t n, int64_t k, const float* d_A, int64_t lda,
                    const float* d_B, int64_t ldb, float* d_C, int64_t ldc, const float* d_bias, int32_t epi,
                    const float* d_mask, int64_t ldmask, void* d_ws, size_t* ws_bytes, hipStream_t stream) {
  g_err.clear();
  if (op < GCN_OP_NN || op > GCN_OP_TN) return fail(GCN_E_INVALID, "gcn_gemm: unknown op");
  if (m < 0 || n < 0 || k < 0) return fail(GCN_E_INVALID, "gcn_gemm: negative size");
  const bool ta = op == GCN_OP_TN, tb = op == GCN_OP_NT;
  if (lda < (ta ? m : k) || ldb < (tb ? k : n) || ldc < n) return fail(GCN_E_INVALID, "gcn_gemm: pitch too small");
  if (epi < GCN_EPI_NONE || epi > GCN_EPI_MASK) return fail(GCN_E_INVALID, "gcn_gemm: unknown epilogue");
  if (epi == GCN_EPI_MASK && (!d_mask || ldmask < n)) return fail(GCN_E_INVALID, "gcn_gemm: mask missing");
  GemmParams p = gemm(m, n, k, d_A, lda, ta, d_B, ldb, tb, d_C, ldc);
  p.bias = d_bias;
  p.epi = epi == GCN_EPI_RELU ? GEMM_RELU : (epi == GCN_EPI_MASK ? GEMM_MASK : GEMM_NONE);
  p.mask = d_mask;
  p.ldmask = ldmask;
  bool query = false;
  GCN_TRY(ws_protocol(d_ws, ws_bytes, gemm_workspace(p), "gcn_gemm", &query));
  if (query) return GCN_OK;
  if (m > 0 && n > 0 && (!d_C || (k > 0 && (!d_A || !d_B)))) return fail(GCN_E_INVALID, "gcn_gemm: NULL operand");
  if (gemm_split_k(p) && p.epi != GEMM_NONE)
    return fail(GCN_E_UNSUPPORTED, "gcn_gemm: split-k launches support only the bias epilogue");
  return launch_gemm(p, d_ws, stream);
}

gcn_status gcn_spmm(int64_t nrows, int64_t nnz, const int64_t* d_ptr, const int32_t* d_idx,
                    const float* d_val, int64_t b_rows, int32_t w, const float* d_B, int64_t ldb,
                    float* d_C, int64_t ldc, const gcn_split* split, void* d_ws, size_t* ws_bytes,
                    hipStream_t stream) {
  g_err.clear();
  if (nrows < 0 || nrows > INT32_MAX || w < 0 || b_rows < 0 || ldb < w || ldc < w)
    return fail(GCN_E_INVALID, "gcn_spmm: bad size or pitch");
  if (split && split->rows && split->n_long > 0 && (!split->first || !split->owner))
    return fail(GCN_E_INVALID, "gcn_spmm: split plan arrays missing");
  bool query = false;
  GCN_TRY(ws_protocol(d_ws, ws_bytes, aggregate_workspace(split, w), "gcn_spmm", &query));
  if (query) return GCN_OK;
  if (nrows > 0 && w > 0 && (!d_ptr || !d_idx || !d_val || !d_B || !d_C))
    return fail(GCN_E_INVALID, "gcn_spmm: NULL argument");
  AggParams p{};
  p.n = (int32_t)nrows;
  p.row_ptr = d_ptr;
  p.col = d_idx;
  p.val = d_val;
  p.M = d_B;
  p.ldm = ldb;
  p.w = w;
  p.Z = d_C;
  p.ldz = ldc;
  p.epi = AGG_NONE;
  p.tag = "spmm";
  return launch_aggregate(p, nnz, split, d_ws, stream);
}

gcn_status gcn_spmm_xt(int32_t n, int32_t f, int64_t nnz, const int64_t* d_col_ptr, const int32_t* d_row,
                       const float* d_cval, const gcn_split* csc_split, const float* d_B, int64_t ldb,
                       int32_t w, float* d_C, int64_t ldc, void* d_ws, size_t* ws_bytes, hipStream_t stream) {
  g_err.clear();
  if (n < 0 || f < 0 || nnz < 0 || w < 0 || ldb < w || ldc < w) return fail(GCN_E_INVALID, "gcn_spmm_xt: bad size or pitch");
  if (csc_split && csc_split->rows && csc_split->n_long > 0 && (!csc_split->first || !csc_split->owner))
    return fail(GCN_E_INVALID, "gcn_spmm_xt: split plan arrays missing");
  if (w > 256 && xt_tiled_enabled(n, f, nnz, w)) return fail(GCN_E_UNSUPPORTED, "gcn_spmm_xt: width above 256");
  bool query = false;
  GCN_TRY(ws_protocol(d_ws, ws_bytes, spmm_xt_workspace(n, f, nnz, w, csc_split), "gcn_spmm_xt", &query));
  if (query) return GCN_OK;
  if (f > 0 && w > 0 && (!d_col_ptr || (nnz > 0 && (!d_row || !d_cval || !d_B)) || !d_C))
    return fail(GCN_E_INVALID, "gcn_spmm_xt: NULL argument");
  if (f == 0 || w == 0) return GCN_OK;
  return launch_spmm_xt(n, f, nnz, d_col_ptr, d_row, d_cval, csc_split, d_B, ldb, w, d_C, ldc, d_ws, stream);
}

gcn_status gcn_spmm_xw(int32_t n, int32_t f, int64_t nnz, const int64_t* d_row_ptr, const int32_t* d_col,
                       const float* d_val, const float* d_W, int64_t ldw, int32_t w, float* d_C, int64_t ldc,
                       void* d_ws, size_t* ws_bytes, hipStream_t stream) {
  g_err.clear();
  if (n < 0 || f < 0 || nnz < 0 || w < 0 || ldw < w || ldc < w) return fail(GCN_E_INVALID, "gcn_spmm_xw: bad size or pitch");
  bool query = false;
  GCN_TRY(ws_protocol(d_ws, ws_bytes, 0, "gcn_spmm_xw", &query));
  if (query) return GCN_OK;
  if (n > 0 && w > 0 && (!d_row_ptr || (nnz > 0 && (!d_col || !d_val || !d_W)) || !d_C))
    return fail(GCN_E_INVALID, "gcn_spmm_xw: NULL argument");
  if (n == 0 || w == 0) return GCN_OK;
  return launch_spmm_xw(n, nnz, d_row_ptr, d_col, d_val, d_W, ldw, w, d_C, ldc, stream);
}

gcn_status gcn_column_sums(int64_t rows, int32_t w, const float* d_G, int64_t ldg, float* d_out,
                           const float* d_row_vals, float* d_mean, void* d_ws, size_t* ws_bytes,
                           hipStream_t stream) {
  g_err.clear();
  if (rows < 0 || w < 0 || ldg < w) return fail(GCN_E_INVALID, "gcn_column_sums: bad size or pitch");
  bool query = false;
  GCN_TRY(ws_protocol(d_ws, ws_bytes, colsum_workspace(rows, w), "gcn_column_sums", &query));
  if (query) return GCN_OK;
  if ((w > 0 && (!d_out || (rows > 0 && !d_G))) || (d_row_vals && !d_mean) || (rows > 0 && d_mean && !d_row_vals))
    return fail(GCN_E_INVALID, "gcn_column_sums: NULL argument");
  return launch_colsum(rows, w, d_G, ldg, d_out, d_row_vals, d_mean, d_ws, stream);
}

gcn_status gcn_adam(const gcn_adam_tensor* t, int32_t count, int32_t step, double lr, double beta1,
                    double beta2, double eps, hipStream_t stream) {
  g_err.clear();
  if (count < 0 || (count > 0 && !t) || step < 1) return fail(GCN_E_INVALID, "gcn_adam: bad arguments");
  for (int i = 0; i < count; ++i)
    if (t[i].count < 0 || (t[i].count > 0 && (!t[i].param || !t[i].grad || !t[i].m || !t[i].v)))
      return fail(GCN_E_INVALID, "gcn_adam: bad tensor");
  return launch_adam(t, count, step, nullptr, lr, beta1, beta2, eps, stream);
}

gcn_status gcn_adam_device_step(const gcn_adam_tensor* t, int32_t count, int32_t* d_step, double lr,
                                double beta1, double beta2, double eps, hipStream_t stream) {
  g_err.clear();
  if (count < 0 || (count > 0 && !t) || !d_step) return fail(GCN_E_INVALID, "gcn_adam_device_step: bad arguments");
  for (int i = 0; i < count; ++i)
    if (t[i].count < 0 || (t[i].count > 0 && (!t[i].param || !t[i].grad || !t[i].m || !t[i].v)))
      return fail(GCN_E_INVALID, "gcn_adam_device_step: bad tensor");
  return launch_adam(t, count, 1, d_step, lr, beta1, beta2, eps, stream);
}

}  // extern "C"
