// C ABI of the DiT step library: argument validation, the weight manifest,
// the workspace plan and the launch sequence of one denoising step.  All
// device work is enqueued on the caller's stream; nothing here allocates
// device memory or synchronises the host.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <map>
#include <mutex>
#include <string>
#include <tuple>
#include <vector>

#include "dit_internal.h"

using namespace dit;

namespace {

thread_local std::string g_err;

dit_status fail(dit_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

#define HIP_TRY(expr)                                                                      \
  do {                                                                                     \
    hipError_t e_ = (expr);                                                                \
    if (e_ != hipSuccess) return fail(DIT_ERR_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// ---------------------------------------------------------------------------- kernel timing
struct ProfFamily {
  std::string name;
  long launches = 0;
  double ms = 0, flops = 0, bytes = 0;
};
struct ProfRecord {
  int family;
  hipEvent_t begin, end;
  double flops, bytes;
};
struct Profiler {
  std::recursive_mutex mu;  // timed() nests for the per-shape detail entries
  bool on = false;
  std::vector<hipEvent_t> pool;
  size_t used = 0;
  std::vector<ProfRecord> recs;
  std::vector<ProfFamily> fams;
};
Profiler& prof() {
  static Profiler* p = new Profiler();
  return *p;
}

hipError_t prof_event(hipEvent_t* ev) {
  Profiler& P = prof();
  if (P.used == P.pool.size()) {
    hipEvent_t e;
    hipError_t err = hipEventCreate(&e);
    if (err != hipSuccess) return err;
    P.pool.push_back(e);
  }
  *ev = P.pool[P.used++];
  return hipSuccess;
}

// Runs one launch; when profiling is on, brackets it with events on stream s.
template <class F>
hipError_t timed(hipStream_t s, const char* family, double flops, double bytes, F&& launch) {
  Profiler& P = prof();
  if (!P.on) return launch();
  std::lock_guard<std::recursive_mutex> lock(P.mu);
  int fi = -1;
  for (size_t i = 0; i < P.fams.size(); ++i)
    if (P.fams[i].name == family) fi = (int)i;
  if (fi < 0) {
    P.fams.push_back(ProfFamily());
    P.fams.back().name = family;
    fi = (int)P.fams.size() - 1;
  }
  ProfRecord r;
  r.family = fi;
  r.flops = flops;
  r.bytes = bytes;
  hipError_t e;
  if ((e = prof_event(&r.begin)) != hipSuccess || (e = prof_event(&r.end)) != hipSuccess) return e;
  if ((e = hipEventRecord(r.begin, s)) != hipSuccess) return e;
  hipError_t le = launch();
  if ((e = hipEventRecord(r.end, s)) != hipSuccess) return e;
  P.recs.push_back(r);
  return le;
}

int elem_size(int dtype) { return dtype == DIT_BF16 ? 2 : 4; }

// ---------------------------------------------------------------------------- validation
dit_status check_config(const dit_config* c) {
  if (!c) return fail(DIT_ERR_INVALID_ARG, "config is NULL");
  if (c->dtype != DIT_F32 && c->dtype != DIT_BF16) return fail(DIT_ERR_INVALID_ARG, "dtype %d", c->dtype);
  if (c->hidden <= 0 || c->heads <= 0 || c->head_dim <= 0 || c->heads * c->head_dim != c->hidden)
    return fail(DIT_ERR_INVALID_ARG, "hidden %d != heads %d * head_dim %d", c->hidden, c->heads, c->head_dim);
  if (c->hidden % 64 != 0 || c->hidden > 4096)
    return fail(DIT_ERR_UNSUPPORTED, "hidden %d must be a multiple of 64 and <= 4096", c->hidden);
  if (c->dtype == DIT_BF16 && c->head_dim != 128 && c->head_dim != 64)
    return fail(DIT_ERR_UNSUPPORTED, "bf16 models need head_dim 128 or 64 (got %d)", c->head_dim);
  if (c->dtype == DIT_F32 && c->head_dim != 64)
    return fail(DIT_ERR_UNSUPPORTED, "fp32 models need head_dim 64 (got %d)", c->head_dim);
  if (c->mlp_ratio <= 0 || c->mlp_ratio > 8) return fail(DIT_ERR_INVALID_ARG, "mlp_ratio %d", c->mlp_ratio);
  if (c->n_double < 0 || c->n_single < 0 || c->n_double + c->n_single > 1024)
    return fail(DIT_ERR_INVALID_ARG, "block counts %d / %d", c->n_double, c->n_single);
  if (c->in_channels <= 0 || c->in_channels % 8 != 0)
    return fail(DIT_ERR_UNSUPPORTED, "in_channels %d must be a positive multiple of 8", c->in_channels);
  if (c->text_dim <= 0 || c->text_dim % 8 != 0)
    return fail(DIT_ERR_UNSUPPORTED, "text_dim %d must be a positive multiple of 8", c->text_dim);
  if (c->time_freq_dim <= 0 || c->time_freq_dim % 8 != 0 || c->time_freq_dim > 4096)
    return fail(DIT_ERR_UNSUPPORTED, "time_freq_dim %d must be a positive multiple of 8, at most 4096",
                c->time_freq_dim);
  if (!(c->rope_theta > 0.f) || !(c->ln_eps > 0.f))
    return fail(DIT_ERR_INVALID_ARG, "rope_theta and ln_eps must be positive");
  if (c->flags & ~DIT_FLAG_BATCH_INVARIANT) return fail(DIT_ERR_INVALID_ARG, "unknown flags 0x%x", c->flags);
  return DIT_OK;
}

dit_status check_batch(const dit_batch* b, bool need_t) {
  if (!b) return fail(DIT_ERR_INVALID_ARG, "batch is NULL");
  if (b->n_req < 1 || b->n_req > DIT_MAX_REQUESTS)
    return fail(DIT_ERR_INVALID_ARG, "n_req %d outside [1, %d]", b->n_req, DIT_MAX_REQUESTS);
  if (!b->grid_h || !b->grid_w || !b->n_txt) return fail(DIT_ERR_INVALID_ARG, "batch arrays are NULL");
  if (need_t && !b->t) return fail(DIT_ERR_INVALID_ARG, "batch timesteps are NULL");
  long total = 0;
  for (int r = 0; r < b->n_req; ++r) {
    if (b->grid_h[r] < 1 || b->grid_h[r] > DIT_MAX_GRID || b->grid_w[r] < 1 || b->grid_w[r] > DIT_MAX_GRID)
      return fail(DIT_ERR_INVALID_ARG, "request %d grid %dx%d outside [1, %d]", r, b->grid_h[r], b->grid_w[r],
                  DIT_MAX_GRID);
    if (b->n_txt[r] < 0 || b->n_txt[r] > (1 << 20))
      return fail(DIT_ERR_INVALID_ARG, "request %d n_txt %d", r, b->n_txt[r]);
    if (need_t && !(b->t[r] >= 0.f && b->t[r] <= 1.f))
      return fail(DIT_ERR_INVALID_ARG, "request %d timestep %g outside [0, 1]", r, (double)b->t[r]);
    total += (long)b->grid_h[r] * b->grid_w[r] + b->n_txt[r];
  }
  if (total > (1L << 24)) return fail(DIT_ERR_UNSUPPORTED, "batch of %ld tokens is too large", total);
  return DIT_OK;
}

BatchMeta make_meta(const dit_batch* b) {
  BatchMeta m{};
  m.n_req = b->n_req;
  for (int r = 0; r < b->n_req; ++r) {
    const int ni = b->grid_h[r] * b->grid_w[r], nt = b->n_txt[r];
    m.txt_off[r + 1] = m.txt_off[r] + nt;
    m.img_off[r + 1] = m.img_off[r] + ni;
    m.joint_off[r + 1] = m.joint_off[r] + nt + ni;
    m.pad_off[r + 1] = m.pad_off[r] + (nt + ni + kSeqPad - 1) / kSeqPad * kSeqPad;
    m.n_txt[r] = nt;
    m.grid_w[r] = b->grid_w[r];
  }
  m.T_txt = m.txt_off[b->n_req];
  m.T_img = m.img_off[b->n_req];
  m.T = m.T_txt + m.T_img;
  return m;
}

// ---------------------------------------------------------------------------- model layout
struct Layout {
  int H, F, d, heads, ns, mod_rows;
  int n_double, n_single;
  // parameter indices in manifest order
  int dbl(int i, int stream /*0 img, 1 txt*/) const { return 10 + (i * ns + (ns == 2 ? stream : 0)) * 8; }
  int sgl(int i) const { return 10 + n_double * ns * 8 + i * 4; }
  int fin() const { return 10 + n_double * ns * 8 + n_single * 4; }
  int count() const { return fin() + 2; }
  // modulation row offsets
  int mod_dbl(int i, int stream) const { return (i * ns + (ns == 2 ? stream : 0)) * 6 * H; }
  int mod_sgl(int i) const { return n_double * ns * 6 * H + i * 3 * H; }
  int mod_fin() const { return n_double * ns * 6 * H + n_single * 3 * H; }
};

Layout make_layout(const dit_config* c) {
  Layout l;
  l.H = c->hidden;
  l.F = c->mlp_ratio * c->hidden;
  l.d = c->head_dim;
  l.heads = c->heads;
  l.ns = c->tie_streams ? 1 : 2;
  l.n_double = c->n_double;
  l.n_single = c->n_single;
  l.mod_rows = (c->n_double * l.ns * 6 + c->n_single * 3 + 2) * c->hidden;
  return l;
}

struct ManifestEntry {
  std::string name;
  int ndim;
  int shape[2];
};

std::vector<ManifestEntry> build_manifest(const dit_config* c) {
  const Layout L = make_layout(c);
  const int H = L.H, F = L.F;
  std::vector<ManifestEntry> v;
  auto add2 = [&](const std::string& n, int a, int b) { v.push_back({n, 2, {a, b}}); };
  auto add1 = [&](const std::string& n, int a) { v.push_back({n, 1, {a, 0}}); };
  add2("time_in.w1", H, c->time_freq_dim);
  add1("time_in.b1", H);
  add2("time_in.w2", H, H);
  add1("time_in.b2", H);
  add2("img_in.w", H, c->in_channels);
  add1("img_in.b", H);
  add2("txt_in.w", H, c->text_dim);
  add1("txt_in.b", H);
  add2("mod.w", L.mod_rows, H);
  add1("mod.b", L.mod_rows);
  const char* sn[2] = {"img", "txt"};
  for (int i = 0; i < c->n_double; ++i)
    for (int s = 0; s < L.ns; ++s) {
      const std::string p = "double." + std::to_string(i) + "." + sn[s] + ".";
      add2(p + "qkv.w", 3 * H, H);
      add1(p + "qkv.b", 3 * H);
      add2(p + "proj.w", H, H);
      add1(p + "proj.b", H);
      add2(p + "mlp1.w", F, H);
      add1(p + "mlp1.b", F);
      add2(p + "mlp2.w", H, F);
      add1(p + "mlp2.b", H);
    }
  for (int i = 0; i < c->n_single; ++i) {
    const std::string p = "single." + std::to_string(i) + ".";
    add2(p + "lin1.w", 3 * H + F, H);
    add1(p + "lin1.b", 3 * H + F);
    add2(p + "lin2.w", H, H + F);
    add1(p + "lin2.b", H);
  }
  add2("final.w", c->in_channels, H);
  add1("final.b", c->in_channels);
  return v;
}

// ---------------------------------------------------------------------------- workspace
struct Workspace {
  float* mods;   // [n_req, mod_rows]
  float* temb;   // [n_req, tf]
  float* u;      // [n_req, H]
  float* cvec;   // [n_req, H]
  float2* rope;  // [DIT_MAX_GRID, d/4]
  float* X;      // [T, H] residual stream
  void* A;       // [T, H] LayerNorm output, row pitch lda
  void* Q;       // [heads, Tp, d]
  void* K;       // [heads, Tp, d]
  void* Vt;      // [heads, d, Tp], row pitch ldvt
  void* Z;       // [T, H + F]  attention output | MLP hidden, row pitch ldz
  long lda, ldz, ldvt;  // row pitches in elements (see kRowPad)
  float* sk_part;  // partial sums of split GEMMs (kSplitPartBytes), null when GEMMs never split
  int* sk_cnt;     // their arrival counters [kSplitMaxTiles], zeroed at the start of every call
  size_t bytes;
};

// Row pitches of the activations that GEMMs and attention stream (A, Z, V^T)
// are padded by 64 elements past their width.  With unpadded pitches (6 KB,
// 30 KB, 9 KB, 33 KB ...: multiples of 4 KB or of 2 KB) the rows of one
// operand tile fall on few L2 channels; the padding spreads them.
constexpr long kRowPad = 64;

Workspace plan_workspace(const dit_config* c, const BatchMeta& m, char* base) {
  const Layout L = make_layout(c);
  const int es = elem_size(c->dtype);
  const size_t T = m.T, Tp = m.pad_off[m.n_req], n = m.n_req;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char* p = base ? base + off : nullptr;
    off += align256(bytes);
    return (void*)p;
  };
  Workspace w;
  w.mods = (float*)take(n * L.mod_rows * 4);
  w.temb = (float*)take(n * c->time_freq_dim * 4);
  w.u = (float*)take(n * L.H * 4);
  w.cvec = (float*)take(n * L.H * 4);
  w.rope = (float2*)take((size_t)DIT_MAX_GRID * (L.d / 4) * sizeof(float2));
  w.X = (float*)take(T * L.H * 4);
  w.lda = L.H + kRowPad;
  w.ldz = L.H + L.F + kRowPad;
  w.ldvt = (long)Tp + kRowPad;
  w.A = take(T * w.lda * es);
  w.Q = take((size_t)L.heads * Tp * L.d * es);
  w.K = take((size_t)L.heads * Tp * L.d * es);
  w.Vt = take((size_t)L.heads * L.d * w.ldvt * es);
  w.Z = take(T * (size_t)w.ldz * es);
  const bool split = c->dtype == DIT_BF16 && !(c->flags & DIT_FLAG_BATCH_INVARIANT);
  w.sk_part = split ? (float*)take(kSplitPartBytes) : nullptr;
  w.sk_cnt = split ? (int*)take(kSplitMaxTiles * sizeof(int)) : nullptr;
  w.bytes = off;
  return w;
}

// ---------------------------------------------------------------------------- execution context
struct Ctx {
  const dit_config* c;
  Layout L;
  BatchMeta meta;
  const void* const* W;
  Workspace ws;
  hipStream_t s;
  int es;
};

double gemm_flops(const GemmProblem& p) {
  double f = 0;
  for (int g = 0; g < p.n_groups; ++g) f += 2.0 * p.g[g].M * (double)p.N * p.g[g].K;
  return f;
}

// operands read once, output written once (fp32 residual updates read and write)
double gemm_bytes(const GemmProblem& p, int es) {
  double b = 0;
  for (int g = 0; g < p.n_groups; ++g) {
    const GemmGroup& G = p.g[g];
    const int oes = (G.epi.mode == EPI_STORE_F32 || G.epi.mode == EPI_RESID) ? 4 : es;
    b += (double)G.M * G.K * es + (double)p.N * G.K * es + (double)G.M * p.N * oes;
    if (G.epi.mode == EPI_RESID) b += (double)G.M * p.N * 4;
  }
  return b;
}

const char* epi_name(int mode) {
  static const char* n[] = {"store_f32", "store", "gelu", "resid", "qkv"};
  return (mode >= 0 && mode <= 4) ? n[mode] : "?";
}

hipError_t gemm(hipStream_t s, int dtype, const GemmProblem& p) {
  const int es = dtype == DIT_BF16 ? 2 : 4;
  if (dtype == DIT_BF16 && gemm_bf16_split_groups(p)) {
    GemmProblem q = p;
    q.n_groups = 1;
    const hipError_t e = gemm(s, dtype, q);
    if (e != hipSuccess) return e;
    q.g[0] = p.g[1];
    return gemm(s, dtype, q);
  }
  if (dtype == DIT_BF16) {
    if (!prof().on)
      return launch_gemm_bf16(p, s);
    // kernel family for the roofline, plus a per-shape entry ("detail:" prefix)
    // that splits the same launches by N, K and epilogue
    char detail[160];
    int M = p.g[0].M + (p.n_groups > 1 ? p.g[1].M : 0);
    snprintf(detail, sizeof(detail), "detail:%s M=%d N=%d K=%d %s", gemm_bf16_config_name(p), M, p.N, p.g[0].K,
             epi_name(p.g[0].epi.mode));
    hipError_t e = hipSuccess;
    hipError_t r = timed(s, detail, gemm_flops(p), gemm_bytes(p, es), [&] {
      e = timed(s, gemm_bf16_config_name(p), gemm_flops(p), gemm_bytes(p, es), [&] { return launch_gemm_bf16(p, s); });
      return e;
    });
    return r != hipSuccess ? r : e;
  }
  return timed(s, "gemm_f32", gemm_flops(p), gemm_bytes(p, es), [&] { return launch_gemm_f32(p, s); });
}

hipError_t gemm(const Ctx& x, const GemmProblem& p) { return gemm(x.s, x.c->dtype, p); }

double attn_flops(const BatchMeta& m, int heads, int d) {
  double f = 0;
  for (int r = 0; r < m.n_req; ++r) {
    const double L = m.joint_off[r + 1] - m.joint_off[r];
    f += 4.0 * L * L * d * heads;
  }
  return f;
}

hipError_t attn_launch(hipStream_t s, int dtype, const AttnArgs& a) {
  const double bytes = 4.0 * a.meta.T * (double)a.heads * a.head_dim * (dtype == DIT_BF16 ? 2 : 4);
  if (dtype == DIT_BF16)
    return timed(s, "attention_bf16", attn_flops(a.meta, a.heads, a.head_dim), bytes,
                 [&] { return launch_attention_bf16(a, s); });
  return timed(s, "attention_f32", attn_flops(a.meta, a.heads, a.head_dim), bytes,
               [&] { return launch_attention_f32(a, s); });
}

hipError_t ln_mod(const Ctx& x, const float* X, int row_begin, int row_end, const float* mods, int mods_ld,
                  int sh_t, int sc_t, int sh_i, int sc_i, void* out) {
  const int H = x.L.H;
  const double bytes = (double)(row_end - row_begin) * H * (4 + x.es);
  return timed(x.s, "ln_modulate", 0.0, bytes, [&] {
    return launch_ln_modulate(x.c->dtype, X, H, row_begin, row_end, x.meta, mods, mods_ld, sh_t, sc_t, sh_i, sc_i,
                              x.c->ln_eps, out, x.ws.lda, x.s);
  });
}

hipError_t gemv(hipStream_t s, int dtype, const void* W, const void* b, const float* xin, long ldx, int n_req, int K,
                int N, int act, float* y, long ldy) {
  const int es = dtype == DIT_BF16 ? 2 : 4;
  const double bytes = (double)N * K * es + (double)N * es + 4.0 * n_req * ((double)K + N);
  return timed(s, "gemv", 2.0 * n_req * (double)N * K, bytes,
               [&] { return launch_gemv(dtype, W, b, xin, ldx, n_req, K, N, act, y, ldy, s); });
}

EpiArgs epi_base(int mode, int row_base) {
  EpiArgs e;
  memset(&e, 0, sizeof(e));
  e.mode = mode;
  e.row_base = row_base;
  return e;
}

GemmGroup group(const void* A, long lda, const void* W, long ldw, int M, int K, const EpiArgs& e) {
  GemmGroup g;
  g.A = A;
  g.lda = lda;
  g.W = W;
  g.ldw = ldw;
  g.M = M;
  g.K = K;
  g.epi = e;
  return g;
}

// Adds group g to problem p unless it has no rows.
void add_group(GemmProblem& p, const GemmGroup& g) {
  if (g.M > 0) p.g[p.n_groups++] = g;
}

GemmProblem problem(const Ctx& x, int N) {
  GemmProblem p;
  memset(&p, 0, sizeof(p));
  p.N = N;
  p.meta = x.meta;
  p.sk_part = x.ws.sk_part;
  p.sk_cnt = x.ws.sk_cnt;
  return p;
}

const char* elem_ptr(const void* base, long elems, int es) { return (const char*)base + elems * es; }

EpiArgs epi_qkv(const Ctx& x, int row_base) {
  EpiArgs e = epi_base(EPI_QKV, row_base);
  e.q = x.ws.Q;
  e.k = x.ws.K;
  e.vt = x.ws.Vt;
  e.T = x.meta.pad_off[x.meta.n_req];
  e.vt_ld = x.ws.ldvt;
  e.hidden = x.L.H;
  e.head_dim = x.L.d;
  e.n_qkv = 3 * x.L.H;
  e.rope = x.ws.rope;
  e.gelu_out = (char*)x.ws.Z + (long)row_base * x.ws.ldz * x.es;
  e.gelu_ld = x.ws.ldz;
  e.gelu_col0 = x.L.H;
  return e;
}

EpiArgs epi_resid(const Ctx& x, float* X, int row_base, const float* mods, int mods_ld, int gate_off) {
  EpiArgs e = epi_base(EPI_RESID, row_base);
  e.out = X + (long)row_base * x.L.H;
  e.ldo = x.L.H;
  e.mods = mods;
  e.mods_ld = mods_ld;
  e.gate_off = gate_off;
  return e;
}

hipError_t attention(const Ctx& x) {
  AttnArgs a;
  memset(&a, 0, sizeof(a));
  const long Tp = x.meta.pad_off[x.meta.n_req];
  a.q = x.ws.Q;
  a.q_tok = x.L.d;
  a.q_head = Tp * x.L.d;
  a.k = x.ws.K;
  a.k_tok = x.L.d;
  a.k_head = Tp * x.L.d;
  a.vt = x.ws.Vt;
  a.vt_head = (long)x.L.d * x.ws.ldvt;
  a.vt_d = x.ws.ldvt;
  a.o = x.ws.Z;
  a.o_tok = x.ws.ldz;
  a.o_head = x.L.d;
  a.o_stream_major = 1;
  a.heads = x.L.heads;
  a.head_dim = x.L.d;
  a.scale = 1.0f / sqrtf((float)x.L.d);
  for (int r = 0; r <= x.meta.n_req; ++r) a.qk_off[r] = a.vt_off[r] = x.meta.pad_off[r];
  a.meta = x.meta;
  // the split GEMMs' partial-sum slots double as the attention's key-split
  // scratch (the two never run at once); null in batch-invariant mode
  if (x.ws.sk_part && attn_split_bytes(x.meta, a.heads, a.head_dim) <= (size_t)kSplitPartBytes)
    a.split_buf = x.ws.sk_part;
  return attn_launch(x.s, x.c->dtype, a);
}

const void* Wt(const Ctx& x, int idx) { return x.W[idx]; }

// One double-stream block on x.ws.X-like residual `X`.  mods: [n_req, mods_ld];
// off_img / off_txt: each stream's 6H modulation chunk offsets.
dit_status run_double(const Ctx& x, int i, float* X, const float* mods, int mods_ld, int off_img, int off_txt) {
  const int H = x.L.H, F = x.L.F, Tt = x.meta.T_txt, Ti = x.meta.T_img, T = x.meta.T, es = x.es;
  const int bi = x.L.dbl(i, 0), bt = x.L.dbl(i, 1);
  const float eps = x.c->ln_eps;
  const long ldz = x.ws.ldz, lda = x.ws.lda;
  // 1. adaLN (shift1, scale1)
  HIP_TRY(ln_mod(x, X, 0, T, mods, mods_ld, off_txt, off_txt + H, off_img, off_img + H, x.ws.A));
  // 2. QKV projections (+ RoPE on image rows), scattered into the joint Q/K/V^T layout
  {
    GemmProblem p = problem(x, 3 * H);
    EpiArgs et = epi_qkv(x, 0), ei = epi_qkv(x, Tt);
    et.bias = Wt(x, bt + 1);
    ei.bias = Wt(x, bi + 1);
    add_group(p, group(x.ws.A, lda, Wt(x, bt), H, Tt, H, et));
    add_group(p, group(elem_ptr(x.ws.A, (long)Tt * lda, es), lda, Wt(x, bi), H, Ti, H, ei));
    HIP_TRY(gemm(x, p));
  }
  // 3. joint attention -> Z[:, 0:H]
  HIP_TRY(attention(x));
  // 4. output projection + gated residual (gate1)
  {
    GemmProblem p = problem(x, H);
    EpiArgs et = epi_resid(x, X, 0, mods, mods_ld, off_txt + 2 * H);
    EpiArgs ei = epi_resid(x, X, Tt, mods, mods_ld, off_img + 2 * H);
    et.bias = Wt(x, bt + 3);
    ei.bias = Wt(x, bi + 3);
    add_group(p, group(x.ws.Z, ldz, Wt(x, bt + 2), H, Tt, H, et));
    add_group(p, group(elem_ptr(x.ws.Z, (long)Tt * ldz, es), ldz, Wt(x, bi + 2), H, Ti, H, ei));
    HIP_TRY(gemm(x, p));
  }
  // 5. adaLN (shift2, scale2)
  HIP_TRY(ln_mod(x, X, 0, T, mods, mods_ld, off_txt + 3 * H, off_txt + 4 * H, off_img + 3 * H, off_img + 4 * H,
                 x.ws.A));
  // 6. MLP up + GELU -> Z[:, H:H+F]
  {
    GemmProblem p = problem(x, F);
    EpiArgs et = epi_base(EPI_GELU, 0), ei = epi_base(EPI_GELU, Tt);
    et.out = x.ws.Z;
    ei.out = (char*)x.ws.Z + (long)Tt * ldz * es;
    et.ldo = ei.ldo = ldz;
    et.col0 = ei.col0 = H;
    et.bias = Wt(x, bt + 5);
    ei.bias = Wt(x, bi + 5);
    add_group(p, group(x.ws.A, lda, Wt(x, bt + 4), H, Tt, H, et));
    add_group(p, group(elem_ptr(x.ws.A, (long)Tt * lda, es), lda, Wt(x, bi + 4), H, Ti, H, ei));
    HIP_TRY(gemm(x, p));
  }
  // 7. MLP down + gated residual (gate2)
  {
    GemmProblem p = problem(x, H);
    EpiArgs et = epi_resid(x, X, 0, mods, mods_ld, off_txt + 5 * H);
    EpiArgs ei = epi_resid(x, X, Tt, mods, mods_ld, off_img + 5 * H);
    et.bias = Wt(x, bt + 7);
    ei.bias = Wt(x, bi + 7);
    add_group(p, group(elem_ptr(x.ws.Z, H, es), ldz, Wt(x, bt + 6), F, Tt, F, et));
    add_group(p, group(elem_ptr(x.ws.Z, (long)Tt * ldz + H, es), ldz, Wt(x, bi + 6), F, Ti, F, ei));
    HIP_TRY(gemm(x, p));
  }
  return DIT_OK;
}

// Rows of an M x N GEMM (N a multiple of 256) that fill whole rounds of
// 256 x 256 tiles on the 256 CUs, when the rest would leave a last round at
// most a quarter full (0: no such split).  At 2048 px the single blocks'
// linear2 (16 896 x 3072) is 16 384 rows in 3 rounds and a 24-tile remainder.
int full_round_rows(int M, int N) {
  constexpr int kCUs = 256, kTile = 256;
  if (N % kTile != 0) return 0;
  const int tn = N / kTile;
  int unit = 1;  // row tiles per whole number of rounds: 256 / gcd(tn, 256)
  while ((unit * tn) % kCUs != 0) ++unit;
  const long rows_unit = (long)unit * kTile;
  const long M1 = (M / rows_unit) * rows_unit;
  const long rest_tiles = (long)((M - M1 + kTile - 1) / kTile) * tn;
  if (M1 == 0 || M1 == M || 4 * rest_tiles > kCUs) return 0;
  return (int)M1;
}

dit_status run_single(const Ctx& x, int i, float* X, const float* mods, int mods_ld, int off) {
  const int H = x.L.H, F = x.L.F, T = x.meta.T;
  const int b = x.L.sgl(i);
  const long ldz = x.ws.ldz;
  HIP_TRY(ln_mod(x, X, 0, T, mods, mods_ld, off, off + H, off, off + H, x.ws.A));
  {
    GemmProblem p = problem(x, 3 * H + F);
    EpiArgs e = epi_qkv(x, 0);
    e.bias = Wt(x, b + 1);
    add_group(p, group(x.ws.A, x.ws.lda, Wt(x, b), H, T, H, e));
    HIP_TRY(gemm(x, p));
  }
  HIP_TRY(attention(x));
  {
    // Rows [0, T1) form whole rounds of 256 x 256 tiles; a short remainder
    // [T1, T) becomes a second group, which the launch model may run as a
    // launch of its own with K split across the otherwise idle CUs.
    GemmProblem p = problem(x, H);
    const int T1 = full_round_rows(T, H);
    EpiArgs e = epi_resid(x, X, 0, mods, mods_ld, off + 2 * H);
    e.bias = Wt(x, b + 3);
    add_group(p, group(x.ws.Z, ldz, Wt(x, b + 2), H + F, T1 > 0 ? T1 : T, H + F, e));
    if (T1 > 0) {
      EpiArgs e2 = epi_resid(x, X, T1, mods, mods_ld, off + 2 * H);
      e2.bias = Wt(x, b + 3);
      add_group(p, group(elem_ptr(x.ws.Z, (long)T1 * ldz, x.es), ldz, Wt(x, b + 2), H + F, T - T1, H + F, e2));
    }
    HIP_TRY(gemm(x, p));
  }
  return DIT_OK;
}

dit_status check_weights(const dit_config* c, const dit_weights* w) {
  if (!w || !w->tensors) return fail(DIT_ERR_INVALID_ARG, "weights are NULL");
  const int n = make_layout(c).count();
  if (w->n_tensors != n) return fail(DIT_ERR_INVALID_ARG, "expected %d weight tensors, got %d", n, w->n_tensors);
  for (int i = 0; i < n; ++i) {
    if (!w->tensors[i]) return fail(DIT_ERR_INVALID_ARG, "weight tensor %d is NULL", i);
    if (((uintptr_t)w->tensors[i]) % 16 != 0) return fail(DIT_ERR_INVALID_ARG, "weight tensor %d is not 16-byte aligned", i);
  }
  return DIT_OK;
}

dit_status check_ws(void* ws, size_t ws_bytes, size_t need) {
  if (!ws) return fail(DIT_ERR_WORKSPACE, "workspace is NULL");
  if (((uintptr_t)ws) % 256 != 0) return fail(DIT_ERR_WORKSPACE, "workspace is not 256-byte aligned");
  if (ws_bytes < need) return fail(DIT_ERR_WORKSPACE, "workspace %zu bytes < required %zu", ws_bytes, need);
  return DIT_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p) % 16 == 0; }

// ---------------------------------------------------------------------------- static scratch
// Workspace of dit_step_noalloc, for callers that cannot allocate device
// memory (graph capture, serving loops that forbid it).  Every GPU the
// library runs on holds its own copy until the process ends; calls on one GPU
// share it, so calls that overlap on one GPU race.  The step clears what must
// start at zero (split-K counters, the padding of V^T) itself.  In host code
// `scratch` names a host-side stand-in: kernels receive the device address
// from noalloc_scratch, never the symbol.
constexpr size_t kNoAllocScratchBytes = DIT_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;
__device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

// Device address of `scratch` on the device that runs `stream` (the current
// device for the null stream), looked up once per device with that device
// current.
dit_status noalloc_scratch(hipStream_t stream, void** out) {
  static std::mutex mu;
  static void* table[kMaxDevices] = {};
  int cur = 0, dev = 0;
  HIP_TRY(hipGetDevice(&cur));
  dev = cur;
  if (stream) HIP_TRY(hipStreamGetDevice(stream, &dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(DIT_ERR_UNSUPPORTED, "device %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(mu);
  if (!table[dev]) {
    if (dev != cur) HIP_TRY(hipSetDevice(dev));
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (dev != cur) HIP_TRY(hipSetDevice(cur));
    if (e != hipSuccess) return fail(DIT_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    if (!p || ((uintptr_t)p) % 256 != 0) return fail(DIT_ERR_HIP, "static scratch address %p is not usable", p);
    table[dev] = p;
  }
  *out = table[dev];
  return DIT_OK;
}
// Host validation of a dit_step call; fills the batch metadata and the
// workspace bytes the step needs.  Enqueues nothing.
dit_status check_step(const dit_config* cfg, const dit_weights* w, const dit_batch* batch, const void* latents,
                      const void* text_emb, const void* velocity, BatchMeta* meta, size_t* need) {
  dit_status st;
  if ((st = check_config(cfg)) || (st = check_batch(batch, true)) || (st = check_weights(cfg, w))) return st;
  *meta = make_meta(batch);
  if (!latents || !velocity || (meta->T_txt > 0 && !text_emb))
    return fail(DIT_ERR_INVALID_ARG, "latents / text_emb / velocity is NULL");
  if (!aligned16(latents) || !aligned16(velocity) || (text_emb && !aligned16(text_emb)))
    return fail(DIT_ERR_INVALID_ARG, "latents / text_emb / velocity must be 16-byte aligned");
  *need = plan_workspace(cfg, *meta, nullptr).bytes;
  return DIT_OK;
}

// The launch sequence of one denoising step on a validated call; `ws` holds
// at least the planned workspace.
dit_status run_step(const dit_config* cfg, const dit_weights* w, const dit_batch* batch, const BatchMeta& meta,
                    const void* latents, const void* text_emb, void* velocity, void* ws, void* stream) {
  dit_status st;
  Ctx x;
  x.c = cfg;
  x.L = make_layout(cfg);
  x.meta = meta;
  x.W = w->tensors;
  x.ws = plan_workspace(cfg, meta, (char*)ws);
  x.s = (hipStream_t)stream;
  x.es = elem_size(cfg->dtype);
  const int H = x.L.H, n = meta.n_req;
  const int dt = cfg->dtype;

  // conditioning: c = W2 SiLU(W1 e(t) + b1) + b2; all modulation vectors m = Wm SiLU(c) + bm
  HIP_TRY(timed(x.s, "setup", 0.0, 0.0, [&] { return launch_rope_table(x.ws.rope, x.L.d, cfg->rope_theta, x.s); }));
  HIP_TRY(timed(x.s, "setup", 0.0, 0.0,
                [&] { return launch_zero_i32(x.ws.sk_cnt, x.ws.sk_cnt ? kSplitMaxTiles : 0, x.s); }));
  HIP_TRY(timed(x.s, "setup", 0.0, 0.0,
                [&] { return launch_vt_pad_zero(dt, x.ws.Vt, x.ws.ldvt, meta, x.L.heads, x.L.d, x.s); }));
  HIP_TRY(timed(x.s, "setup", 0.0, 0.0,
                [&] { return launch_timestep_embed(x.ws.temb, n, batch->t, cfg->time_freq_dim, x.s); }));
  HIP_TRY(gemv(x.s, dt, Wt(x, 0), Wt(x, 1), x.ws.temb, cfg->time_freq_dim, n, cfg->time_freq_dim, H, 0, x.ws.u, H));
  HIP_TRY(gemv(x.s, dt, Wt(x, 2), Wt(x, 3), x.ws.u, H, n, H, H, 1, x.ws.cvec, H));
  HIP_TRY(gemv(x.s, dt, Wt(x, 8), Wt(x, 9), x.ws.cvec, H, n, H, x.L.mod_rows, 1, x.ws.mods, x.L.mod_rows));

  // input embedders -> residual stream X (stream-major rows)
  {
    GemmProblem p = problem(x, H);
    EpiArgs et = epi_base(EPI_STORE_F32, 0), ei = epi_base(EPI_STORE_F32, meta.T_txt);
    et.out = x.ws.X;
    ei.out = x.ws.X + (long)meta.T_txt * H;
    et.ldo = ei.ldo = H;
    et.bias = Wt(x, 7);
    ei.bias = Wt(x, 5);
    add_group(p, group(text_emb, cfg->text_dim, Wt(x, 6), cfg->text_dim, meta.T_txt, cfg->text_dim, et));
    add_group(p, group(latents, cfg->in_channels, Wt(x, 4), cfg->in_channels, meta.T_img, cfg->in_channels, ei));
    HIP_TRY(gemm(x, p));
  }
  for (int i = 0; i < cfg->n_double; ++i)
    if ((st = run_double(x, i, x.ws.X, x.ws.mods, x.L.mod_rows, x.L.mod_dbl(i, 0), x.L.mod_dbl(i, 1)))) return st;
  for (int i = 0; i < cfg->n_single; ++i)
    if ((st = run_single(x, i, x.ws.X, x.ws.mods, x.L.mod_rows, x.L.mod_sgl(i)))) return st;

  // final layer on the image rows -> velocity
  const int off = x.L.mod_fin();
  HIP_TRY(ln_mod(x, x.ws.X, meta.T_txt, meta.T, x.ws.mods, x.L.mod_rows, off, off + H, off, off + H, x.ws.A));
  {
    const int fb = x.L.fin();
    GemmProblem p = problem(x, cfg->in_channels);
    EpiArgs e = epi_base(EPI_STORE_T, meta.T_txt);
    e.out = velocity;
    e.ldo = cfg->in_channels;
    e.bias = Wt(x, fb + 1);
    add_group(p, group(x.ws.A, x.ws.lda, Wt(x, fb), H, meta.T_img, H, e));
    HIP_TRY(gemm(x, p));
  }
  return DIT_OK;
}


}  // namespace

// ============================================================================ C ABI
extern "C" {

const char* dit_last_error(void) { return g_err.c_str(); }

dit_status dit_weight_count(const dit_config* cfg, int* count) {
  g_err.clear();
  dit_status st = check_config(cfg);
  if (st) return st;
  if (!count) return fail(DIT_ERR_INVALID_ARG, "count is NULL");
  *count = make_layout(cfg).count();
  return DIT_OK;
}

dit_status dit_weight_manifest(const dit_config* cfg, int index, const char** name, int shape[2], int* ndim) {
  g_err.clear();
  dit_status st = check_config(cfg);
  if (st) return st;
  if (!name || !shape || !ndim) return fail(DIT_ERR_INVALID_ARG, "output pointers are NULL");
  static std::mutex mu;
  static std::map<std::vector<int>, std::vector<ManifestEntry>>* cache =
      new std::map<std::vector<int>, std::vector<ManifestEntry>>();
  const std::vector<int> key = {cfg->hidden,      cfg->heads,       cfg->head_dim, cfg->mlp_ratio, cfg->n_double,
                                cfg->n_single,    cfg->in_channels, cfg->text_dim, cfg->time_freq_dim,
                                cfg->tie_streams ? 1 : 0};
  std::lock_guard<std::mutex> lock(mu);
  auto it = cache->find(key);
  if (it == cache->end()) it = cache->emplace(key, build_manifest(cfg)).first;
  const std::vector<ManifestEntry>& m = it->second;
  if (index < 0 || index >= (int)m.size())
    return fail(DIT_ERR_INVALID_ARG, "index %d outside [0, %d)", index, (int)m.size());
  *name = m[index].name.c_str();
  *ndim = m[index].ndim;
  shape[0] = m[index].shape[0];
  shape[1] = m[index].shape[1];
  return DIT_OK;
}

dit_status dit_workspace_size(const dit_config* cfg, const dit_batch* batch, size_t* bytes) {
  g_err.clear();
  dit_status st = check_config(cfg);
  if (st) return st;
  st = check_batch(batch, false);
  if (st) return st;
  if (!bytes) return fail(DIT_ERR_INVALID_ARG, "bytes is NULL");
  const BatchMeta m = make_meta(batch);
  *bytes = plan_workspace(cfg, m, nullptr).bytes;
  return DIT_OK;
}

dit_status dit_step(const dit_config* cfg, const dit_weights* w, const dit_batch* batch, const void* latents,
                    const void* text_emb, void* velocity, void* ws, size_t ws_bytes, void* stream) {
  g_err.clear();
  dit_status st;
  BatchMeta meta;
  size_t need = 0;
  if ((st = check_step(cfg, w, batch, latents, text_emb, velocity, &meta, &need))) return st;
  if ((st = check_ws(ws, ws_bytes, need))) return st;
  return run_step(cfg, w, batch, meta, latents, text_emb, velocity, ws, stream);
}

dit_status dit_step_noalloc(const dit_config* cfg, const dit_weights* w, const dit_batch* batch,
                            const void* latents, const void* text_emb, void* velocity, void* stream) {
  g_err.clear();
  dit_status st;
  BatchMeta meta;
  size_t need = 0;
  if ((st = check_step(cfg, w, batch, latents, text_emb, velocity, &meta, &need))) return st;
  if (need > kNoAllocScratchBytes)
    return fail(DIT_ERR_WORKSPACE, "dit_step_noalloc: this batch needs %zu bytes of workspace, more than the "
                "%zu bytes of the library's static scratch (use dit_step with a caller workspace)",
                need, (size_t)kNoAllocScratchBytes);
  void* ws = nullptr;
  if ((st = noalloc_scratch((hipStream_t)stream, &ws))) return st;
  return run_step(cfg, w, batch, meta, latents, text_emb, velocity, ws, stream);
}

dit_status dit_block_forward(const dit_config* cfg, const dit_weights* w, int kind, int index,
                             const dit_batch* batch, float* hidden, const float* cond, void* ws, size_t ws_bytes,
                             void* stream) {
  g_err.clear();
  dit_status st;
  if ((st = check_config(cfg)) || (st = check_batch(batch, false)) || (st = check_weights(cfg, w))) return st;
  if (kind != 0 && kind != 1) return fail(DIT_ERR_INVALID_ARG, "kind %d (0 double, 1 single)", kind);
  if (index < 0 || index >= (kind == 0 ? cfg->n_double : cfg->n_single))
    return fail(DIT_ERR_INVALID_ARG, "block index %d out of range", index);
  if (!hidden || !cond) return fail(DIT_ERR_INVALID_ARG, "hidden / cond is NULL");
  if (!aligned16(hidden) || !aligned16(cond)) return fail(DIT_ERR_INVALID_ARG, "hidden / cond must be 16-byte aligned");
  const BatchMeta meta = make_meta(batch);
  const Workspace need = plan_workspace(cfg, meta, nullptr);
  if ((st = check_ws(ws, ws_bytes, need.bytes))) return st;

  Ctx x;
  x.c = cfg;
  x.L = make_layout(cfg);
  x.meta = meta;
  x.W = w->tensors;
  x.ws = plan_workspace(cfg, meta, (char*)ws);
  x.s = (hipStream_t)stream;
  x.es = elem_size(cfg->dtype);
  const int H = x.L.H, n = meta.n_req;
  HIP_TRY(timed(x.s, "setup", 0.0, 0.0, [&] { return launch_rope_table(x.ws.rope, x.L.d, cfg->rope_theta, x.s); }));
  HIP_TRY(timed(x.s, "setup", 0.0, 0.0,
                [&] { return launch_zero_i32(x.ws.sk_cnt, x.ws.sk_cnt ? kSplitMaxTiles : 0, x.s); }));
  HIP_TRY(timed(x.s, "setup", 0.0, 0.0,
                [&] { return launch_vt_pad_zero(cfg->dtype, x.ws.Vt, x.ws.ldvt, meta, x.L.heads, x.L.d, x.s); }));
  if (kind == 0) {
    // this block's modulation rows: image stream, then (untied) text stream
    const int off = x.L.mod_dbl(index, 0);
    const int rows = 6 * H * x.L.ns;
    const char* wm = (const char*)Wt(x, 8) + (long)off * H * x.es;
    const char* bm = (const char*)Wt(x, 9) + (long)off * x.es;
    HIP_TRY(gemv(x.s, cfg->dtype, wm, bm, cond, H, n, H, rows, 1, x.ws.mods, rows));
    return run_double(x, index, hidden, x.ws.mods, rows, 0, x.L.ns == 2 ? 6 * H : 0);
  }
  const int off = x.L.mod_sgl(index);
  const char* wm = (const char*)Wt(x, 8) + (long)off * H * x.es;
  const char* bm = (const char*)Wt(x, 9) + (long)off * x.es;
  HIP_TRY(gemv(x.s, cfg->dtype, wm, bm, cond, H, n, H, 3 * H, 1, x.ws.mods, 3 * H));
  return run_single(x, index, hidden, x.ws.mods, 3 * H, 0);
}

dit_status euler_update(const dit_batch* batch, int channels, int dtype, void* latents, const void* velocity,
                        const float* dt, void* stream) {
  g_err.clear();
  dit_status st;
  if ((st = check_batch(batch, false))) return st;
  if (dtype != DIT_F32 && dtype != DIT_BF16) return fail(DIT_ERR_INVALID_ARG, "dtype %d", dtype);
  if (channels <= 0) return fail(DIT_ERR_INVALID_ARG, "channels %d", channels);
  if (!latents || !velocity || !dt) return fail(DIT_ERR_INVALID_ARG, "latents / velocity / dt is NULL");
  for (int r = 0; r < batch->n_req; ++r)
    if (!isfinite(dt[r])) return fail(DIT_ERR_INVALID_ARG, "dt[%d] is not finite", r);
  const BatchMeta meta = make_meta(batch);
  const double bytes = 3.0 * meta.T_img * channels * elem_size(dtype);
  hipStream_t s = (hipStream_t)stream;
  HIP_TRY(timed(s, "euler", 0.0, bytes, [&] { return launch_euler(dtype, latents, velocity, channels, meta, dt, s); }));
  return DIT_OK;
}

dit_status dit_attention_workspace_size(const dit_batch* batch, int heads, int head_dim, int dtype, size_t* bytes) {
  g_err.clear();
  dit_status st;
  if ((st = check_batch(batch, false))) return st;
  if (!bytes) return fail(DIT_ERR_INVALID_ARG, "bytes is NULL");
  if (heads <= 0 || head_dim <= 0) return fail(DIT_ERR_INVALID_ARG, "heads %d head_dim %d", heads, head_dim);
  if (dtype != DIT_F32 && dtype != DIT_BF16) return fail(DIT_ERR_INVALID_ARG, "dtype %d", dtype);
  const BatchMeta m = make_meta(batch);
  *bytes = align256((size_t)heads * head_dim * m.pad_off[m.n_req] * elem_size(dtype));
  if (dtype == DIT_BF16) *bytes += align256(attn_split_bytes(m, heads, head_dim));
  return DIT_OK;
}

dit_status dit_attention(const dit_batch* batch, int heads, int head_dim, int dtype, const void* q, const void* k,
                         const void* v, void* o, void* ws, size_t ws_bytes, void* stream) {
  g_err.clear();
  dit_status st;
  if ((st = check_batch(batch, false))) return st;
  if (dtype != DIT_F32 && dtype != DIT_BF16) return fail(DIT_ERR_INVALID_ARG, "dtype %d", dtype);
  if (heads <= 0) return fail(DIT_ERR_INVALID_ARG, "heads %d", heads);
  if ((dtype == DIT_BF16 && head_dim != 128 && head_dim != 64) || (dtype == DIT_F32 && head_dim != 64))
    return fail(DIT_ERR_UNSUPPORTED, "head_dim %d with dtype %d", head_dim, dtype);
  if (!q || !k || !v || !o) return fail(DIT_ERR_INVALID_ARG, "q / k / v / o is NULL");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o))
    return fail(DIT_ERR_INVALID_ARG, "q / k / v / o must be 16-byte aligned");
  const BatchMeta m = make_meta(batch);
  size_t need = 0;
  dit_attention_workspace_size(batch, heads, head_dim, dtype, &need);
  if ((st = check_ws(ws, ws_bytes, need))) return st;
  hipStream_t s = (hipStream_t)stream;
  HIP_TRY(timed(s, "v_transpose", 0.0, 2.0 * m.T * heads * head_dim * elem_size(dtype),
                [&] { return launch_v_transpose(dtype, v, m, heads, head_dim, ws, s); }));
  HIP_TRY(timed(s, "v_transpose", 0.0, 0.0, [&] { return launch_vt_pad_zero(dtype, ws, m.pad_off[m.n_req], m, heads, head_dim, s); }));
  AttnArgs a;
  memset(&a, 0, sizeof(a));
  const long Tp = m.pad_off[m.n_req];
  a.q = q;
  a.q_tok = (long)heads * head_dim;
  a.q_head = head_dim;
  a.k = k;
  a.k_tok = (long)heads * head_dim;
  a.k_head = head_dim;
  a.vt = ws;
  a.vt_head = (long)head_dim * Tp;
  a.vt_d = Tp;
  a.o = o;
  a.o_tok = (long)heads * head_dim;
  a.o_head = head_dim;
  a.o_stream_major = 0;
  a.heads = heads;
  a.head_dim = head_dim;
  a.scale = 1.0f / sqrtf((float)head_dim);
  for (int r = 0; r <= m.n_req; ++r) {
    a.qk_off[r] = m.joint_off[r];
    a.vt_off[r] = m.pad_off[r];
  }
  a.meta = m;
  if (dtype == DIT_BF16 && attn_split_bytes(m, heads, head_dim) > 0)
    a.split_buf = (float*)((char*)ws + align256((size_t)heads * head_dim * Tp * elem_size(dtype)));
  HIP_TRY(attn_launch(s, dtype, a));
  return DIT_OK;
}

dit_status dit_linear(int M, int N, int K, int dtype, const void* x, const void* w, const void* b, void* y,
                      int out_dtype, void* stream) {
  g_err.clear();
  if (M < 0 || N <= 0 || K <= 0) return fail(DIT_ERR_INVALID_ARG, "M %d N %d K %d", M, N, K);
  if (dtype != DIT_F32 && dtype != DIT_BF16) return fail(DIT_ERR_INVALID_ARG, "dtype %d", dtype);
  if (out_dtype != DIT_F32 && out_dtype != DIT_BF16) return fail(DIT_ERR_INVALID_ARG, "out_dtype %d", out_dtype);
  if (dtype == DIT_F32 && out_dtype != DIT_F32) return fail(DIT_ERR_UNSUPPORTED, "fp32 GEMM stores fp32 only");
  if (K % 8 != 0) return fail(DIT_ERR_UNSUPPORTED, "K %d must be a multiple of 8", K);
  if ((M > 0 && !x) || !w || (M > 0 && !y)) return fail(DIT_ERR_INVALID_ARG, "x / w / y is NULL");
  if (!aligned16(x) || !aligned16(w)) return fail(DIT_ERR_INVALID_ARG, "x / w must be 16-byte aligned");
  if (M == 0) return DIT_OK;
  GemmProblem p;
  memset(&p, 0, sizeof(p));
  p.N = N;
  p.meta.n_req = 1;
  EpiArgs e = epi_base(out_dtype == DIT_F32 ? EPI_STORE_F32 : EPI_STORE_T, 0);
  e.out = y;
  e.ldo = N;
  e.bias = b;
  p.g[0] = group(x, K, w, K, M, K, e);
  p.n_groups = 1;
  HIP_TRY(gemm((hipStream_t)stream, dtype, p));
  return DIT_OK;
}

dit_status dit_profile_start(void) {
  g_err.clear();
  Profiler& P = prof();
  std::lock_guard<std::recursive_mutex> lock(P.mu);
  P.recs.clear();
  P.fams.clear();
  P.used = 0;
  P.on = true;
  return DIT_OK;
}

dit_status dit_profile_stop(int* n_families) {
  g_err.clear();
  Profiler& P = prof();
  std::lock_guard<std::recursive_mutex> lock(P.mu);
  P.on = false;
  for (const ProfRecord& r : P.recs) {
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(r.end);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.begin, r.end);
    if (e != hipSuccess) return fail(DIT_ERR_HIP, "profile events: %s", hipGetErrorString(e));
    ProfFamily& f = P.fams[r.family];
    f.launches += 1;
    f.ms += ms;
    f.flops += r.flops;
    f.bytes += r.bytes;
  }
  P.recs.clear();
  if (n_families) *n_families = (int)P.fams.size();
  return DIT_OK;
}

dit_status dit_profile_entry(int i, const char** family, long* launches, double* total_ms, double* flops,
                             double* bytes) {
  g_err.clear();
  Profiler& P = prof();
  std::lock_guard<std::recursive_mutex> lock(P.mu);
  if (i < 0 || i >= (int)P.fams.size()) return fail(DIT_ERR_INVALID_ARG, "family %d out of range", i);
  const ProfFamily& f = P.fams[i];
  if (family) *family = f.name.c_str();
  if (launches) *launches = f.launches;
  if (total_ms) *total_ms = f.ms;
  if (flops) *flops = f.flops;
  if (bytes) *bytes = f.bytes;
  return DIT_OK;
}

}  // extern "C"
