// Host runtime behind the C ABI of include/cs.h: model weights arena,
// rollout state and step driver, the DiT launch sequence, profiler, and the
// host-side ranking.  Every device computation is one of the kernels in
// k_*.hip; this file only validates, allocates and launches.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <memory>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/cs.h"
#include "kernels.hpp"

using namespace cs;

// ------------------------------------------------------------------ errors
static thread_local std::string g_err;

static cs_status fail(cs_status code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

#define HIPC(call)                                                                   \
  do {                                                                               \
    hipError_t e_ = (call);                                                          \
    if (e_ != hipSuccess) {                                                          \
      if (e_ == hipErrorOutOfMemory)                                                 \
        return fail(CS_E_NOMEM, "%s: %s", #call, hipGetErrorString(e_));            \
      return fail(CS_E_DEVICE, "%s: %s (%d)", #call, hipGetErrorString(e_), (int)e_); \
    }                                                                                \
  } while (0)

#define CHECK(cond, code, ...)                 \
  do {                                         \
    if (!(cond)) return fail(code, __VA_ARGS__); \
  } while (0)

#define GUARD(...)                                                         \
  try {                                                                    \
    __VA_ARGS__                                                            \
  } catch (const std::bad_alloc&) {                                        \
    return fail(CS_E_NOMEM, "host allocation failed");                     \
  } catch (...) {                                                          \
    return fail(CS_E_DEVICE, "unexpected exception in the runtime");       \
  }

// Test hook: cap on device bytes a single allocation may request (0 = none),
// so that out-of-memory handling can be exercised without exhausting HBM.
static size_t g_alloc_cap = 0;
extern "C" void cs_debug_set_alloc_cap(size_t bytes) { g_alloc_cap = bytes; }

static cs_status dmalloc(void** p, size_t bytes) {
  *p = nullptr;
  if (bytes == 0) bytes = 256;
  if (g_alloc_cap && bytes > g_alloc_cap)
    return fail(CS_E_NOMEM, "device allocation of %zu bytes exceeds the test cap", bytes);
  hipError_t e = hipMalloc(p, bytes);
  if (e != hipSuccess) {
    *p = nullptr;
    (void)hipGetLastError();
    return fail(CS_E_NOMEM, "hipMalloc(%zu): %s", bytes, hipGetErrorString(e));
  }
  return CS_OK;
}

#define TRY(x)                    \
  do {                            \
    cs_status s_ = (x);           \
    if (s_ != CS_OK) return s_;   \
  } while (0)

// ---------------------------------------------------------------- profiler
struct Profiler {
  bool on = false;
  struct Rec { int fam; hipEvent_t a, b; };
  std::vector<Rec> recs;
  std::vector<hipEvent_t> pool;
  double total[CS_K_COUNT] = {0};
  long count[CS_K_COUNT] = {0};

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
  void begin(int fam, hipStream_t st, hipEvent_t* out) {
    *out = nullptr;
    if (!on) return;
    hipEvent_t a = get();
    if (a && hipEventRecord(a, st) == hipSuccess) *out = a;
    (void)fam;
  }
  void end(int fam, hipStream_t st, hipEvent_t a) {
    if (!on || !a) return;
    hipEvent_t b = get();
    if (b && hipEventRecord(b, st) == hipSuccess) recs.push_back({fam, a, b});
  }
  void flush() {
    for (auto& r : recs) {
      float ms = 0.0f;
      if (hipEventSynchronize(r.b) == hipSuccess && hipEventElapsedTime(&ms, r.a, r.b) == hipSuccess) {
        total[r.fam] += ms;
        count[r.fam] += 1;
      }
      pool.push_back(r.a);
      pool.push_back(r.b);
    }
    recs.clear();
  }
  void reset() {
    flush();
    for (int i = 0; i < CS_K_COUNT; ++i) { total[i] = 0; count[i] = 0; }
  }
  ~Profiler() {
    for (auto& r : recs) { hipEventDestroy(r.a); hipEventDestroy(r.b); }
    for (auto e : pool) hipEventDestroy(e);
  }
};

struct ProfScope {
  Profiler& p; int fam; hipStream_t st; hipEvent_t a;
  ProfScope(Profiler& p_, int f, hipStream_t s) : p(p_), fam(f), st(s), a(nullptr) { p.begin(fam, st, &a); }
  ~ProfScope() { p.end(fam, st, a); }
};

// ---------------------------------------------------------- weight layout
struct TSpec { std::string name; long rows, cols; bool matrix; };

static std::vector<TSpec> weight_spec(const cs_model_desc& m) {
  const long d = m.hidden, p = (long)m.in_ch * m.patch_t * m.patch_h * m.patch_w, F = m.ffn;
  std::vector<TSpec> s = {
      {"patch_w", d, p, true},   {"patch_b", 1, d, false},
      {"text1_w", d, m.text_dim, true}, {"text1_b", 1, d, false},
      {"text2_w", d, d, true},   {"text2_b", 1, d, false},
      {"time1_w", d, m.freq_dim, true}, {"time1_b", 1, d, false},
      {"time2_w", d, d, true},   {"time2_b", 1, d, false},
      {"mod_w", 6 * d, d, true}, {"mod_b", 1, 6 * d, false},
  };
  for (int j = 0; j < m.n_blocks; ++j) {
    const std::string b = "blk" + std::to_string(j) + ".";
    std::vector<TSpec> blk = {
        {b + "mod", 6, d, false},
        {b + "qkv_w", 3 * d, d, true}, {b + "qkv_b", 1, 3 * d, false},
        {b + "q_gain", 1, d, false}, {b + "k_gain", 1, d, false},
        {b + "o_w", d, d, true}, {b + "o_b", 1, d, false},
        {b + "ca_ln_g", 1, d, false}, {b + "ca_ln_b", 1, d, false},
        {b + "caq_w", d, d, true}, {b + "caq_b", 1, d, false},
        {b + "cak_w", d, d, true}, {b + "cak_b", 1, d, false},
        {b + "cav_w", d, d, true}, {b + "cav_b", 1, d, false},
        {b + "caq_gain", 1, d, false}, {b + "cak_gain", 1, d, false},
        {b + "cao_w", d, d, true}, {b + "cao_b", 1, d, false},
        {b + "ffn1_w", F, d, true}, {b + "ffn1_b", 1, F, false},
        {b + "ffn2_w", d, F, true}, {b + "ffn2_b", 1, d, false},
    };
    s.insert(s.end(), blk.begin(), blk.end());
  }
  s.push_back({"head_mod", 2, d, false});
  s.push_back({"head_w", p, d, true});
  s.push_back({"head_b", 1, p, false});
  return s;
}

static cs_status validate_desc(const cs_model_desc* m) {
  CHECK(m, CS_E_INVAL, "model desc is NULL");
  CHECK(m->n_blocks >= 1 && m->hidden >= 1 && m->heads >= 1 && m->head_dim >= 1 && m->ffn >= 1 &&
            m->text_dim >= 1 && m->text_len >= 1 && m->in_ch >= 1 && m->lat_f >= 1 &&
            m->lat_h >= 1 && m->lat_w >= 1,
        CS_E_INVAL, "model dimensions must be positive");
  CHECK(m->dtype == CS_BF16 || m->dtype == CS_FP32, CS_E_INVAL, "dtype must be CS_BF16 or CS_FP32");
  CHECK(m->hidden == m->heads * m->head_dim, CS_E_INVAL, "hidden != heads * head_dim");
  CHECK(m->head_dim == 32 || m->head_dim == 64 || m->head_dim == 128, CS_E_UNSUPPORTED,
        "head_dim must be 32, 64 or 128");
  CHECK(m->hidden % 64 == 0 && m->ffn % 64 == 0 && m->text_dim % 64 == 0, CS_E_UNSUPPORTED,
        "hidden, ffn and text_dim must be multiples of 64");
  CHECK(m->freq_dim == 256, CS_E_UNSUPPORTED, "freq_dim must be 256");
  CHECK(m->patch_t == 1 && m->patch_h == 2 && m->patch_w == 2, CS_E_UNSUPPORTED,
        "patch must be (1,2,2)");
  CHECK(m->lat_h % 2 == 0 && m->lat_w % 2 == 0, CS_E_INVAL, "lat_h and lat_w must be even");
  CHECK((m->in_ch * 4) % 64 == 0, CS_E_UNSUPPORTED, "in_ch must be a multiple of 16");
  const long L = (long)m->lat_f * (m->lat_h / 2) * (m->lat_w / 2);
  CHECK(L <= (1L << 24), CS_E_UNSUPPORTED, "too many tokens");
  return CS_OK;
}

// ------------------------------------------------------------------ model
struct Block {
  const void *qkv_w, *o_w, *caq_w, *cak_w, *cav_w, *cao_w, *ffn1_w, *ffn2_w;
  const float *qkv_b, *q_gain, *k_gain, *o_b, *ca_ln_g, *ca_ln_b, *caq_b, *cak_b, *cav_b,
      *caq_gain, *cak_gain, *cao_b, *ffn1_b, *ffn2_b;
};

struct Workspace {
  int cap = 0;
  void *patches = nullptr, *u = nullptr, *qk = nullptr, *vt = nullptr, *o = nullptr,
       *q2 = nullptr, *h = nullptr;
  float* z = nullptr;
  int32_t* ids = nullptr;     // identity slot ids [cap] (velocity calls)
  int32_t* zeros = nullptr;   // branch 0 for every slot [cap]
  void release() {
    void* ps[] = {patches, u, qk, vt, o, q2, h, z, ids, zeros};
    for (void* p : ps) if (p) hipFree(p);
    *this = Workspace();
  }
};

struct CtxKV {
  int B = 0;
  void* k = nullptr;    // [blocks][B][Lt][d]
  void* vt = nullptr;   // [blocks][B][d][Ltp]
  void* tmp0 = nullptr; // [Lt][max(text_dim, d)]
  void* tmp1 = nullptr; // [Lt][d]
  void* emb = nullptr;  // [Lt][d]
  void release() {
    void* ps[] = {k, vt, tmp0, tmp1, emb};
    for (void* p : ps) if (p) hipFree(p);
    *this = CtxKV();
  }
};

struct cs_model {
  cs_model_desc desc;
  hipStream_t stream = nullptr;
  size_t esz = 2;        // bytes per matrix element
  long d = 0, L = 0, P = 0, D = 0, Lp = 0, Ltp = 0;
  int gf = 0, gh = 0, gw = 0;
  void* arena = nullptr;
  const void *patch_w, *text1_w, *text2_w, *time1_w, *time2_w, *mod_w, *head_w;
  const float *patch_b, *text1_b, *text2_b, *time1_b, *time2_b, *mod_b, *head_mod, *head_b;
  const float* mod_tables = nullptr;  // [n_blocks][6][d]
  std::vector<Block> blocks;
  float2* rope = nullptr;
  float* cond = nullptr;   // time features, h1, e, m, mods, hmod
  float *tfeat, *h1, *e, *m, *mods, *hmod;
  Profiler prof;
  Workspace vel_ws;
  CtxKV vel_ctx;
  ~cs_model() {
    vel_ws.release();
    vel_ctx.release();
    if (arena) hipFree(arena);
    if (rope) hipFree(rope);
    if (cond) hipFree(cond);
  }
};

struct cs_rollout {
  cs_model* model = nullptr;
  cs_rollout_desc desc;
  std::vector<float> t;
  int S = 0;            // streams = n_cand * n_branch
  long D = 0;
  int nchunk = 0, nschunk = 0;
  float *x = nullptr, *xref = nullptr, *delta = nullptr, *vbuf = nullptr, *wbuf = nullptr;
  float* vtil = nullptr;      // guided velocity of the last step (preview only)
  int vtil_step = -1;         // step whose guided velocity vtil holds
  double *a = nullptr, *partials = nullptr, *spart = nullptr, *scores = nullptr;
  uint8_t *has_ref = nullptr, *ovr = nullptr;
  int32_t *slots = nullptr, *branch = nullptr;
  char* dec = nullptr;        // device decision block: DecideOut | a_seen[S] | mask[S]
  char* dec_host = nullptr;   // pinned mirror
  uint8_t* ovr_host = nullptr;  // pinned staging for override masks
  double* scores_host = nullptr;
  Workspace ws;
  CtxKV ctx;
  int steps_done = 0;
  int decided_step = 0;
  int n_compute = 0;
  // attention-output broadcasting (CS_CACHE_PAB): stored branch outputs
  // [n_blocks][S][L][d] of the compute type, and whether any is stored
  void *pab_self = nullptr, *pab_cross = nullptr;
  bool pab_have_self = false, pab_have_cross = false;
  long long self_reused = 0, cross_reused = 0;
  std::vector<uint8_t> has_ref_h;
  long long calls = 0, computed = 0;
  size_t dec_bytes() const { return sizeof(DecideOut) + (size_t)S * sizeof(double) + (size_t)S; }
  double* a_seen_dev() { return reinterpret_cast<double*>(dec + sizeof(DecideOut)); }
  uint8_t* mask_dev() { return reinterpret_cast<uint8_t*>(dec + sizeof(DecideOut) + (size_t)S * sizeof(double)); }
  const double* a_seen_h() const { return reinterpret_cast<const double*>(dec_host + sizeof(DecideOut)); }
  const uint8_t* mask_h() const { return reinterpret_cast<const uint8_t*>(dec_host + sizeof(DecideOut) + (size_t)S * sizeof(double)); }
  ~cs_rollout() {
    ws.release();
    ctx.release();
    void* ps[] = {x, xref, delta, vbuf, vtil, a, partials, spart, scores, has_ref, ovr, slots, branch, dec,
                  pab_self, pab_cross};
    for (void* p : ps) if (p) hipFree(p);
    if (dec_host) hipHostFree(dec_host);
    if (ovr_host) hipHostFree(ovr_host);
    if (scores_host) hipHostFree(scores_host);
  }
};

// ------------------------------------------------------------- allocation
static cs_status ws_alloc(cs_model* m, Workspace& w, int cap) {
  if (w.cap >= cap) return CS_OK;
  w.release();
  const cs_model_desc& g = m->desc;
  const long rows = (long)cap * m->L;
  const size_t e = m->esz;
  TRY(dmalloc(&w.patches, rows * m->P * e));
  TRY(dmalloc((void**)&w.z, rows * m->d * sizeof(float)));
  TRY(dmalloc(&w.u, rows * m->d * e));
  TRY(dmalloc(&w.qk, rows * 2 * m->d * e));
  TRY(dmalloc(&w.vt, (size_t)cap * m->d * m->Lp * e));
  TRY(dmalloc(&w.o, rows * m->d * e));
  TRY(dmalloc(&w.q2, rows * m->d * e));
  TRY(dmalloc(&w.h, rows * (long)g.ffn * e));
  TRY(dmalloc((void**)&w.ids, cap * sizeof(int32_t)));
  TRY(dmalloc((void**)&w.zeros, cap * sizeof(int32_t)));
  // V^T padding columns must hold finite values (they meet zero weights).
  HIPC(hipMemsetAsync(w.vt, 0, (size_t)cap * m->d * m->Lp * e, m->stream));
  std::vector<int32_t> ids(cap), zeros(cap, 0);
  for (int i = 0; i < cap; ++i) ids[i] = i;
  HIPC(hipMemcpyAsync(w.ids, ids.data(), cap * sizeof(int32_t), hipMemcpyHostToDevice, m->stream));
  HIPC(hipMemcpyAsync(w.zeros, zeros.data(), cap * sizeof(int32_t), hipMemcpyHostToDevice, m->stream));
  HIPC(hipStreamSynchronize(m->stream));
  w.cap = cap;
  return CS_OK;
}

static cs_status ctx_alloc(cs_model* m, CtxKV& c, int B) {
  if (c.B >= B) return CS_OK;
  c.release();
  const cs_model_desc& g = m->desc;
  const size_t e = m->esz;
  const long Lt = g.text_len;
  TRY(dmalloc(&c.k, (size_t)g.n_blocks * B * Lt * m->d * e));
  TRY(dmalloc(&c.vt, (size_t)g.n_blocks * B * m->d * m->Ltp * e));
  TRY(dmalloc(&c.tmp0, (size_t)Lt * std::max<long>(g.text_dim, m->d) * e));
  TRY(dmalloc(&c.tmp1, (size_t)Lt * m->d * e));
  TRY(dmalloc(&c.emb, (size_t)Lt * m->d * e));
  HIPC(hipMemsetAsync(c.vt, 0, (size_t)g.n_blocks * B * m->d * m->Ltp * e, m->stream));
  c.B = B;
  return CS_OK;
}

// ---------------------------------------------------------- DiT sequence
template <typename T>
static cs_status build_ctx(cs_model* m, CtxKV& c, int b, const float* ctx) {
  const cs_model_desc& g = m->desc;
  hipStream_t st = m->stream;
  const long Lt = g.text_len, d = m->d;
  ProfScope ps(m->prof, CS_K_OTHER, st);
  T* tmp0 = (T*)c.tmp0;
  T* tmp1 = (T*)c.tmp1;
  T* emb = (T*)c.emb;
  HIPC(cast_from_f32<T>(ctx, tmp0, Lt * g.text_dim, st));
  HIPC(gemm_store<T>(tmp0, g.text_dim, (const T*)m->text1_w, (int)Lt, (int)d, g.text_dim,
                     m->text1_b, 1, tmp1, d, st));
  HIPC(gemm_store<T>(tmp1, d, (const T*)m->text2_w, (int)Lt, (int)d, (int)d, m->text2_b, 0, emb, d, st));
  for (int j = 0; j < g.n_blocks; ++j) {
    const Block& bk = m->blocks[j];
    T* K = (T*)c.k + ((long)j * c.B + b) * Lt * d;
    T* VT = (T*)c.vt + ((long)j * c.B + b) * d * m->Ltp;
    HIPC(gemm_store<T>(emb, d, (const T*)bk.cak_w, (int)Lt, (int)d, (int)d, bk.cak_b, 0, K, d, st));
    HIPC(rmsnorm_rope<T>(K, Lt, d, (int)d, 1, bk.cak_gain, nullptr, nullptr, 1, g.head_dim, st));
    HIPC(gemm_store_t<T>(emb, d, (const T*)bk.cav_w, (int)Lt, (int)d, (int)d, bk.cav_b, VT, m->Ltp, st));
  }
  return CS_OK;
}

// Time conditioning for timestep t: e, m, per-block modulation, head modulation.
template <typename T>
static cs_status time_cond(cs_model* m, float t) {
  const cs_model_desc& g = m->desc;
  hipStream_t st = m->stream;
  const int d = (int)m->d;
  ProfScope ps(m->prof, CS_K_OTHER, st);
  HIPC(time_features(t, g.freq_dim, m->tfeat, st));
  HIPC(gemv<T>((const T*)m->time1_w, m->tfeat, m->time1_b, d, g.freq_dim, 0, m->h1, st));
  HIPC(gemv<T>((const T*)m->time2_w, m->h1, m->time2_b, d, d, 1, m->e, st));
  HIPC(gemv<T>((const T*)m->mod_w, m->e, m->mod_b, 6 * d, d, 1, m->m, st));
  HIPC(build_mods_strided(m->m, m->e, m->mod_tables, 6L * d, g.n_blocks, m->head_mod, d, m->mods,
                          m->hmod, st));
  return CS_OK;
}

// Attention-output broadcasting for one transformer evaluation: per branch,
// COMPUTE (no store), STORE (compute and keep the output) or REUSE (apply the
// kept output).  The arrays are [n_blocks][n_slots][L][d]; rows follow the
// evaluation's row order, so the slots must be the same streams in the same
// order on every call of a rollout.
enum PabMode { PAB_COMPUTE = 0, PAB_STORE = 1, PAB_REUSE = 2 };
struct PabIO {
  void* self_y; void* cross_y;
  int self_mode, cross_mode;
};

// One transformer evaluation for n_slots streams.  Stream s reads latent
// x + (slot_id[s] / cand_div) * D, attends to text branch kv_branch[s], and
// writes its velocity to vout + slot_id[s] * D.
template <typename T>
static cs_status dit_forward(cs_model* m, Workspace& w, CtxKV& c, const float* x,
                             const int32_t* slot_id, const int32_t* kv_branch, int n_slots,
                             int cand_div, float t, float* vout, const PabIO* pab) {
  const cs_model_desc& g = m->desc;
  hipStream_t st = m->stream;
  Profiler& pf = m->prof;
  const long L = m->L, d = m->d, rows = (long)n_slots * L;
  const int F = g.ffn, H = g.heads;
  const float sl2 = (float)(1.4426950408889634 / sqrt((double)g.head_dim));
  T* U = (T*)w.u;
  T* QK = (T*)w.qk;
  T* VT = (T*)w.vt;
  T* O = (T*)w.o;
  T* Q2 = (T*)w.q2;
  T* Hh = (T*)w.h;
  float* Z = w.z;

  TRY(time_cond<T>(m, t));
  {
    ProfScope ps(pf, CS_K_GEMM, st);
    HIPC(patchify<T>(x, slot_id, n_slots, cand_div, m->D, g.in_ch, g.lat_f, g.lat_h, g.lat_w,
                     (T*)w.patches, st));
    HIPC(gemm_patch<T>((const T*)w.patches, (const T*)m->patch_w, (int)rows, (int)d, (int)m->P,
                       m->patch_b, Z, st));
  }
  const int self_mode = pab ? pab->self_mode : PAB_COMPUTE;
  const int cross_mode = pab ? pab->cross_mode : PAB_COMPUTE;
  for (int j = 0; j < g.n_blocks; ++j) {
    const Block& bk = m->blocks[j];
    const float* md = m->mods + (long)j * 6 * d;
    T* y_self = pab ? (T*)pab->self_y + (long)j * rows * d : nullptr;
    T* y_cross = pab ? (T*)pab->cross_y + (long)j * rows * d : nullptr;
    // self-attention
    if (self_mode == PAB_REUSE) {
      ProfScope ps(pf, CS_K_OTHER, st);
      HIPC(residual_add<T>(Z, y_self, md + 2 * d, rows, (int)d, st));
    } else {
    { ProfScope ps(pf, CS_K_NORM, st);
      HIPC(layer_norm_mod<T>(Z, rows, (int)d, md + 0 * d, md + 1 * d, 0, U, st)); }
    { ProfScope ps(pf, CS_K_GEMM, st);
      HIPC(gemm_qkv<T>(U, (const T*)bk.qkv_w, (int)rows, (int)d, bk.qkv_b, (int)L, QK, VT, m->Lp, st)); }
    { ProfScope ps(pf, CS_K_NORM, st);
      HIPC(rmsnorm_rope<T>(QK, rows, 2 * d, (int)d, 2, bk.q_gain, bk.k_gain, m->rope, (int)L,
                           g.head_dim, st)); }
    {
      ProfScope ps(pf, CS_K_SELF_ATTN, st);
      AttnArgs<T> a;
      a.q = QK; a.q_ld = 2 * d; a.q_ss = L * 2 * d;
      a.k = QK + d; a.k_ld = 2 * d; a.k_ss = L * 2 * d;
      a.vt = VT; a.vt_ld = m->Lp; a.vt_ss = d * m->Lp;
      a.kv_sel = nullptr;
      a.o = O; a.o_ld = d; a.o_ss = L * d;
      a.lq = (int)L; a.lk = (int)L; a.heads = H; a.n_streams = n_slots; a.scale_log2 = sl2;
      HIPC(flash_attention<T>(a, g.head_dim, st));
    }
    { ProfScope ps(pf, CS_K_GEMM, st);
      HIPC(gemm_residual<T>(O, d, (const T*)bk.o_w, (int)rows, (int)d, (int)d, bk.o_b, md + 2 * d, Z,
                            self_mode == PAB_STORE ? y_self : nullptr, st)); }
    }
    // cross-attention
    if (cross_mode == PAB_REUSE) {
      ProfScope ps(pf, CS_K_OTHER, st);
      HIPC(residual_add<T>(Z, y_cross, nullptr, rows, (int)d, st));
    } else {
    { ProfScope ps(pf, CS_K_NORM, st);
      HIPC(layer_norm_mod<T>(Z, rows, (int)d, bk.ca_ln_g, bk.ca_ln_b, 1, U, st)); }
    { ProfScope ps(pf, CS_K_GEMM, st);
      HIPC(gemm_store<T>(U, d, (const T*)bk.caq_w, (int)rows, (int)d, (int)d, bk.caq_b, 0, Q2, d, st)); }
    { ProfScope ps(pf, CS_K_NORM, st);
      HIPC(rmsnorm_rope<T>(Q2, rows, d, (int)d, 1, bk.caq_gain, nullptr, nullptr, (int)L, g.head_dim, st)); }
    {
      ProfScope ps(pf, CS_K_CROSS_ATTN, st);
      AttnArgs<T> a;
      a.q = Q2; a.q_ld = d; a.q_ss = L * d;
      a.k = (const T*)c.k + (long)j * c.B * g.text_len * d; a.k_ld = d; a.k_ss = (long)g.text_len * d;
      a.vt = (const T*)c.vt + (long)j * c.B * d * m->Ltp; a.vt_ld = m->Ltp; a.vt_ss = d * m->Ltp;
      a.kv_sel = kv_branch;
      a.o = O; a.o_ld = d; a.o_ss = L * d;
      a.lq = (int)L; a.lk = g.text_len; a.heads = H; a.n_streams = n_slots; a.scale_log2 = sl2;
      HIPC(flash_attention<T>(a, g.head_dim, st));
    }
    { ProfScope ps(pf, CS_K_GEMM, st);
      HIPC(gemm_residual<T>(O, d, (const T*)bk.cao_w, (int)rows, (int)d, (int)d, bk.cao_b, nullptr, Z,
                            cross_mode == PAB_STORE ? y_cross : nullptr, st)); }
    }
    // feed-forward
    { ProfScope ps(pf, CS_K_NORM, st);
      HIPC(layer_norm_mod<T>(Z, rows, (int)d, md + 3 * d, md + 4 * d, 0, U, st)); }
    { ProfScope ps(pf, CS_K_GEMM, st);
      HIPC(gemm_store<T>(U, d, (const T*)bk.ffn1_w, (int)rows, F, (int)d, bk.ffn1_b, 1, Hh, F, st));
      HIPC(gemm_residual<T>(Hh, F, (const T*)bk.ffn2_w, (int)rows, (int)d, F, bk.ffn2_b, md + 5 * d, Z,
                            nullptr, st)); }
  }
  { ProfScope ps(pf, CS_K_NORM, st);
    HIPC(layer_norm_mod<T>(Z, rows, (int)d, m->hmod, m->hmod + d, 0, U, st)); }
  { ProfScope ps(pf, CS_K_GEMM, st);
    HIPC(gemm_head<T>(U, (const T*)m->head_w, (int)rows, (int)d, (int)m->P, m->head_b, vout, slot_id,
                      (int)L, m->gh, m->gw, g.lat_f, g.lat_h, g.lat_w, m->D, st)); }
  return CS_OK;
}

static cs_status dit_dispatch(cs_model* m, Workspace& w, CtxKV& c, const float* x,
                              const int32_t* slot_id, const int32_t* kv_branch, int n_slots,
                              int cand_div, float t, float* vout, const PabIO* pab = nullptr) {
  if (m->desc.dtype == CS_BF16)
    return dit_forward<bf16>(m, w, c, x, slot_id, kv_branch, n_slots, cand_div, t, vout, pab);
  return dit_forward<float>(m, w, c, x, slot_id, kv_branch, n_slots, cand_div, t, vout, pab);
}

static cs_status ctx_dispatch(cs_model* m, CtxKV& c, int b, const float* ctx) {
  if (m->desc.dtype == CS_BF16) return build_ctx<bf16>(m, c, b, ctx);
  return build_ctx<float>(m, c, b, ctx);
}

// ------------------------------------------------- allocation-free scoring
// Partial sums of cs_score_noalloc live in this file-scope device array (one
// copy per GPU, held until the process ends).  In host code `scratch` only
// names the symbol: its device address is looked up once per device with
// hipGetSymbolAddress and every launch takes that address.
static __device__ __align__(256) double scratch[CS_SCORE_NOALLOC_MAX_PARTIALS];

static constexpr int MAX_DEVICES = 64;
static double* g_scratch_ptr[MAX_DEVICES] = {nullptr};
static std::mutex g_scratch_mu;

// Device address of `scratch` on the current device (looked up on the
// first call made with that device current).
static cs_status scratch_ptr(double** out) {
  int dev = -1;
  HIPC(hipGetDevice(&dev));
  CHECK(dev >= 0 && dev < MAX_DEVICES, CS_E_UNSUPPORTED, "device index %d out of range", dev);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    HIPC(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    CHECK(p, CS_E_DEVICE, "hipGetSymbolAddress returned NULL for the scoring scratch array");
    g_scratch_ptr[dev] = static_cast<double*>(p);
  }
  *out = g_scratch_ptr[dev];
  return CS_OK;
}

// ================================================================ C ABI
extern "C" {

const char* cs_last_error(void) { return g_err.c_str(); }

cs_status cs_model_weight_count(const cs_model_desc* desc, size_t* count) {
  GUARD({
    TRY(validate_desc(desc));
    CHECK(count, CS_E_INVAL, "count is NULL");
    size_t n = 0;
    for (auto& s : weight_spec(*desc)) n += (size_t)(s.rows * s.cols);
    *count = n;
    return CS_OK;
  })
}

static cs_status model_init_impl(const cs_model_desc* desc, const float* weights, size_t n_weights,
                                 void* stream, cs_model** out) {
  TRY(validate_desc(desc));
  CHECK(out, CS_E_INVAL, "out is NULL");
  *out = nullptr;
  CHECK(weights, CS_E_INVAL, "weights is NULL");
  size_t expect = 0;
  auto spec = weight_spec(*desc);
  for (auto& s : spec) expect += (size_t)(s.rows * s.cols);
  CHECK(n_weights == expect, CS_E_INVAL, "weight count %zu, expected %zu", n_weights, expect);

  std::unique_ptr<cs_model> m(new cs_model());
  m->desc = *desc;
  m->stream = (hipStream_t)stream;
  m->esz = desc->dtype == CS_BF16 ? 2 : 4;
  m->d = desc->hidden;
  m->gf = desc->lat_f;
  m->gh = desc->lat_h / 2;
  m->gw = desc->lat_w / 2;
  m->L = (long)m->gf * m->gh * m->gw;
  m->P = (long)desc->in_ch * 4;
  m->D = (long)desc->in_ch * desc->lat_f * desc->lat_h * desc->lat_w;
  const int kvt = attn_kv_tile((int)m->esz, desc->head_dim);
  m->Lp = round_up(m->L, kvt);
  m->Ltp = round_up(desc->text_len, kvt);

  // arena: matrices in the compute type, vectors fp32; block modulation
  // tables gathered into one [n_blocks][6][d] array.  In bf16 the weights of
  // the direct-load GEMM (every matrix except the three time-conditioning
  // GEMV matrices and the narrow head) are stored in its tiled layout.
  auto tiled = [&](const TSpec& t) {
    return m->esz == 2 && t.matrix && t.name != "time1_w" && t.name != "time2_w" &&
           t.name != "mod_w" && t.name != "head_w";
  };
  std::vector<size_t> off(spec.size());
  size_t bytes = 0;
  const size_t tables_bytes = (size_t)desc->n_blocks * 6 * m->d * sizeof(float);
  size_t tables_off = 0;
  bytes = round_up(tables_bytes, 256);
  for (size_t i = 0; i < spec.size(); ++i) {
    const bool is_table = spec[i].name.size() > 4 && spec[i].name.compare(spec[i].name.size() - 4, 4, ".mod") == 0;
    if (is_table) { off[i] = (size_t)-1; continue; }
    off[i] = bytes;
    const long elems = tiled(spec[i]) ? gemm_tiled_weight_elems((int)spec[i].rows, (int)spec[i].cols)
                                      : spec[i].rows * spec[i].cols;
    bytes += round_up((size_t)elems * (spec[i].matrix ? m->esz : 4), 256);
  }
  TRY(dmalloc(&m->arena, bytes));
  char* base = (char*)m->arena;
  hipStream_t st = m->stream;
  size_t src = 0;
  int table_j = 0;
  std::vector<const void*> ptr(spec.size());
  for (size_t i = 0; i < spec.size(); ++i) {
    const long n = spec[i].rows * spec[i].cols;
    if (off[i] == (size_t)-1) {
      float* dst = (float*)(base + tables_off) + (long)table_j * 6 * m->d;
      HIPC(hipMemcpyAsync(dst, weights + src, n * sizeof(float), hipMemcpyDeviceToDevice, st));
      ptr[i] = dst;
      ++table_j;
    } else if (spec[i].matrix) {
      if (tiled(spec[i]))
        HIPC(gemm_tile_weight(weights + src, (int)spec[i].rows, (int)spec[i].cols, (bf16*)(base + off[i]), st));
      else if (m->esz == 2)
        HIPC(cast_from_f32<bf16>(weights + src, (bf16*)(base + off[i]), n, st));
      else
        HIPC(hipMemcpyAsync(base + off[i], weights + src, n * sizeof(float), hipMemcpyDeviceToDevice, st));
      ptr[i] = base + off[i];
    } else {
      HIPC(hipMemcpyAsync(base + off[i], weights + src, n * sizeof(float), hipMemcpyDeviceToDevice, st));
      ptr[i] = base + off[i];
    }
    src += (size_t)n;
  }
  m->mod_tables = (const float*)(base + tables_off);
  size_t k = 0;
  auto P_ = [&]() { return ptr[k++]; };
  auto F_ = [&]() { return (const float*)ptr[k++]; };
  m->patch_w = P_(); m->patch_b = F_();
  m->text1_w = P_(); m->text1_b = F_();
  m->text2_w = P_(); m->text2_b = F_();
  m->time1_w = P_(); m->time1_b = F_();
  m->time2_w = P_(); m->time2_b = F_();
  m->mod_w = P_(); m->mod_b = F_();
  m->blocks.resize(desc->n_blocks);
  for (int j = 0; j < desc->n_blocks; ++j) {
    Block& b = m->blocks[j];
    (void)P_();  // modulation table (gathered above)
    b.qkv_w = P_(); b.qkv_b = F_(); b.q_gain = F_(); b.k_gain = F_();
    b.o_w = P_(); b.o_b = F_();
    b.ca_ln_g = F_(); b.ca_ln_b = F_();
    b.caq_w = P_(); b.caq_b = F_(); b.cak_w = P_(); b.cak_b = F_();
    b.cav_w = P_(); b.cav_b = F_(); b.caq_gain = F_(); b.cak_gain = F_();
    b.cao_w = P_(); b.cao_b = F_();
    b.ffn1_w = P_(); b.ffn1_b = F_(); b.ffn2_w = P_(); b.ffn2_b = F_();
  }
  m->head_mod = F_(); m->head_w = P_(); m->head_b = F_();

  // RoPE table (cos, sin) per token and rotation pair, angles in double.
  {
    const int hp = desc->head_dim / 2;
    const int n_h = desc->head_dim / 6, n_w = n_h, n_f = hp - n_h - n_w;
    std::vector<float2> tab((size_t)m->L * hp);
    for (int f = 0; f < m->gf; ++f)
      for (int h = 0; h < m->gh; ++h)
        for (int w = 0; w < m->gw; ++w) {
          const long tok = ((long)f * m->gh + h) * m->gw + w;
          for (int p = 0; p < hp; ++p) {
            int pos, idx, n;
            if (p < n_f) { pos = f; idx = p; n = n_f; }
            else if (p < n_f + n_h) { pos = h; idx = p - n_f; n = n_h; }
            else { pos = w; idx = p - n_f - n_h; n = n_w; }
            const double ang = (double)pos * pow(10000.0, -(double)idx / (double)n);
            tab[tok * hp + p] = make_float2((float)cos(ang), (float)sin(ang));
          }
        }
    TRY(dmalloc((void**)&m->rope, tab.size() * sizeof(float2)));
    HIPC(hipMemcpyAsync(m->rope, tab.data(), tab.size() * sizeof(float2), hipMemcpyHostToDevice, st));
    HIPC(hipStreamSynchronize(st));
  }
  {
    const long d = m->d;
    const size_t nf = 256 + d + d + 6 * d + (size_t)desc->n_blocks * 6 * d + 2 * d;
    TRY(dmalloc((void**)&m->cond, nf * sizeof(float)));
    m->tfeat = m->cond;
    m->h1 = m->tfeat + 256;
    m->e = m->h1 + d;
    m->m = m->e + d;
    m->mods = m->m + 6 * d;
    m->hmod = m->mods + (long)desc->n_blocks * 6 * d;
  }
  HIPC(hipStreamSynchronize(st));
  *out = m.release();
  return CS_OK;
}

cs_status cs_model_init(const cs_model_desc* desc, const float* weights, size_t n_weights,
                        void* stream, cs_model** out) {
  GUARD({ return model_init_impl(desc, weights, n_weights, stream, out); })
}

void cs_model_free(cs_model* model) {
  if (!model) return;
  hipStreamSynchronize(model->stream);
  delete model;
}

cs_status cs_velocity(cs_model* m, const float* x, int32_t n, float t, const float* ctx, float* v) {
  GUARD({
    CHECK(m, CS_E_INVAL, "model is NULL");
    CHECK(x && ctx && v, CS_E_INVAL, "x, ctx and v must be non-NULL");
    CHECK(n >= 1 && n <= 4096, CS_E_INVAL, "n must be in [1, 4096]");
    CHECK(isfinite(t), CS_E_INVAL, "t must be finite");
    CHECK(x != v, CS_E_INVAL, "v may not alias x");
    TRY(ws_alloc(m, m->vel_ws, n));
    TRY(ctx_alloc(m, m->vel_ctx, 1));
    TRY(ctx_dispatch(m, m->vel_ctx, 0, ctx));
    TRY(dit_dispatch(m, m->vel_ws, m->vel_ctx, x, m->vel_ws.ids, m->vel_ws.zeros, n, 1, t, v));
    return CS_OK;
  })
}

static cs_status validate_rollout(const cs_model* m, const cs_rollout_desc* r) {
  CHECK(r, CS_E_INVAL, "rollout desc is NULL");
  CHECK(r->n_cand >= 1 && r->n_cand <= 1024, CS_E_INVAL, "n_cand must be in [1, 1024]");
  CHECK(r->n_steps >= 1 && r->n_steps <= 100000, CS_E_INVAL, "n_steps must be >= 1");
  CHECK(r->n_branch == 1 || r->n_branch == 2, CS_E_INVAL, "n_branch must be 1 or 2");
  CHECK(r->k_warm >= 0 && r->k_cool >= 0, CS_E_INVAL, "k_warm and k_cool must be >= 0");
  CHECK(r->mode == CS_CACHE_OFF || r->mode == CS_CACHE_ADAPTIVE || r->mode == CS_CACHE_STATIC ||
            r->mode == CS_CACHE_PAB,
        CS_E_INVAL, "unknown cache mode %d", r->mode);
  CHECK(r->mode != CS_CACHE_PAB || (r->pab_self_range >= 1 && r->pab_cross_range >= 1), CS_E_INVAL,
        "pab_self_range and pab_cross_range must be >= 1");
  CHECK(!(r->tau != r->tau) && r->tau >= 0.0f, CS_E_INVAL, "tau must be >= 0 and not NaN");
  CHECK(isfinite(r->guidance), CS_E_INVAL, "guidance must be finite");
  CHECK(r->mode != CS_CACHE_STATIC || r->static_k >= 1, CS_E_INVAL, "static_k must be >= 1");
  CHECK(r->timesteps, CS_E_INVAL, "timesteps is NULL");
  for (int k = 0; k <= r->n_steps; ++k) CHECK(isfinite(r->timesteps[k]), CS_E_INVAL, "timestep %d not finite", k);
  for (int k = 0; k < r->n_steps; ++k)
    CHECK(r->timesteps[k + 1] < r->timesteps[k], CS_E_INVAL, "timesteps must strictly decrease");
  (void)m;
  return CS_OK;
}

static cs_status rollout_init_impl(cs_model* m, const cs_rollout_desc* desc, const float* x1,
                                   const float* ctx_c, const float* ctx_u, cs_rollout** out) {
  CHECK(m, CS_E_INVAL, "model is NULL");
  CHECK(out, CS_E_INVAL, "out is NULL");
  *out = nullptr;
  TRY(validate_rollout(m, desc));
  CHECK(x1 && ctx_c, CS_E_INVAL, "x1 and ctx_cond must be non-NULL");
  CHECK((desc->n_branch == 2) == (ctx_u != nullptr), CS_E_INVAL,
        "ctx_uncond must be given iff n_branch == 2");
  std::unique_ptr<cs_rollout> r(new cs_rollout());
  r->model = m;
  r->desc = *desc;
  r->t.assign(desc->timesteps, desc->timesteps + desc->n_steps + 1);
  r->desc.timesteps = r->t.data();
  r->S = desc->n_cand * desc->n_branch;
  r->D = m->D;
  r->nchunk = decide_chunks(r->D);
  r->nschunk = score_chunks(r->D);
  const long N = desc->n_cand, S = r->S, D = r->D;
  hipStream_t st = m->stream;
  TRY(dmalloc((void**)&r->x, N * D * sizeof(float)));
  TRY(dmalloc((void**)&r->xref, S * D * sizeof(float)));
  TRY(dmalloc((void**)&r->delta, S * D * sizeof(float)));
  TRY(dmalloc((void**)&r->vbuf, S * D * sizeof(float)));
  TRY(dmalloc((void**)&r->a, S * sizeof(double)));
  TRY(dmalloc((void**)&r->partials, S * r->nchunk * 2 * sizeof(double)));
  TRY(dmalloc((void**)&r->spart, N * r->nschunk * sizeof(double)));
  TRY(dmalloc((void**)&r->scores, N * sizeof(double)));
  TRY(dmalloc((void**)&r->has_ref, S));
  TRY(dmalloc((void**)&r->ovr, S));
  TRY(dmalloc((void**)&r->slots, S * sizeof(int32_t)));
  TRY(dmalloc((void**)&r->branch, S * sizeof(int32_t)));
  TRY(dmalloc((void**)&r->dec, r->dec_bytes()));
  HIPC(hipHostMalloc((void**)&r->dec_host, r->dec_bytes(), hipHostMallocDefault));
  HIPC(hipHostMalloc((void**)&r->ovr_host, S, hipHostMallocDefault));
  HIPC(hipHostMalloc((void**)&r->scores_host, N * sizeof(double), hipHostMallocDefault));
  TRY(ws_alloc(m, r->ws, (int)S));
  TRY(ctx_alloc(m, r->ctx, desc->n_branch));
  if (desc->mode == CS_CACHE_PAB) {
    const size_t bytes = (size_t)m->desc.n_blocks * S * m->L * m->d * m->esz;
    TRY(dmalloc(&r->pab_self, bytes));
    TRY(dmalloc(&r->pab_cross, bytes));
  }
  // reset cache state (Alg. 1: reset at the start of every generation)
  HIPC(hipMemcpyAsync(r->x, x1, N * D * sizeof(float), hipMemcpyDeviceToDevice, st));
  HIPC(hipMemsetAsync(r->xref, 0, S * D * sizeof(float), st));
  HIPC(hipMemsetAsync(r->delta, 0, S * D * sizeof(float), st));
  HIPC(hipMemsetAsync(r->a, 0, S * sizeof(double), st));
  HIPC(hipMemsetAsync(r->has_ref, 0, S, st));
  TRY(ctx_dispatch(m, r->ctx, 0, ctx_c));
  if (desc->n_branch == 2) TRY(ctx_dispatch(m, r->ctx, 1, ctx_u));
  HIPC(hipStreamSynchronize(st));
  r->has_ref_h.assign(S, 0);
  *out = r.release();
  return CS_OK;
}

cs_status cs_rollout_init(cs_model* m, const cs_rollout_desc* desc, const float* x1,
                          const float* ctx_c, const float* ctx_u, cs_rollout** out) {
  GUARD({ return rollout_init_impl(m, desc, x1, ctx_c, ctx_u, out); })
}

void cs_rollout_free(cs_rollout* r) {
  if (!r) return;
  hipStreamSynchronize(r->model->stream);
  delete r;
}

static cs_status decide_impl(cs_rollout* r, int32_t step, const uint8_t* ovr, uint8_t* mask_out,
                             double* a_out) {
  CHECK(r, CS_E_INVAL, "rollout is NULL");
  CHECK(step >= 1 && step <= r->desc.n_steps, CS_E_INVAL, "step %d outside 1..%d", step, r->desc.n_steps);
  CHECK(step == r->steps_done + 1, CS_E_STATE, "step %d requested, next step is %d", step, r->steps_done + 1);
  CHECK(r->decided_step != step, CS_E_STATE, "step %d already decided", step);
  CHECK(!(ovr && r->desc.mode == CS_CACHE_PAB), CS_E_UNSUPPORTED,
        "a replay override is not available in CS_CACHE_PAB mode");
  if (ovr) {
    // a skipped call applies the branch's cached residual: there must be one
    // (CS_CACHE_OFF never stores it; before a branch's first computed call
    // nothing is stored)
    for (int s = 0; s < r->S; ++s) {
      if (ovr[s]) continue;
      CHECK(r->desc.mode != CS_CACHE_OFF, CS_E_INVAL,
            "override skips stream %d, but CS_CACHE_OFF keeps no cached residual", s);
      CHECK(r->has_ref_h[s], CS_E_INVAL,
            "override skips stream %d at step %d before its first computed call (no cached residual)", s,
            step);
    }
  }
  cs_model* m = r->model;
  hipStream_t st = m->stream;
  const cs_rollout_desc& d = r->desc;
  const bool window_forced = step <= d.k_warm || step > d.n_steps - d.k_cool;
  bool any_ref = false;
  for (uint8_t h : r->has_ref_h) any_ref |= h != 0;
  const bool need_partials = d.mode == CS_CACHE_ADAPTIVE && !window_forced && any_ref;
  {
    ProfScope ps(m->prof, CS_K_DECIDE, st);
    if (need_partials)
      HIPC(decide_partials(r->x, r->xref, d.n_cand, d.n_branch, r->D, r->partials, st));
    if (ovr) {
      memcpy(r->ovr_host, ovr, r->S);
      HIPC(hipMemcpyAsync(r->ovr, r->ovr_host, r->S, hipMemcpyHostToDevice, st));
    }
    DecideParams p;
    p.n_streams = r->S; p.n_branch = d.n_branch; p.step = step; p.n_steps = d.n_steps;
    p.k_warm = d.k_warm; p.k_cool = d.k_cool; p.mode = d.mode; p.static_k = std::max(1, d.static_k);
    p.nchunk = r->nchunk; p.use_partials = need_partials ? 1 : 0; p.use_override = ovr ? 1 : 0;
    p.tau = (double)d.tau;
    HIPC(decide_finalize(p, r->partials, r->ovr, r->a, r->has_ref, r->mask_dev(), r->a_seen_dev(),
                         r->slots, r->branch, reinterpret_cast<DecideOut*>(r->dec), st));
  }
  HIPC(hipMemcpyAsync(r->dec_host, r->dec, r->dec_bytes(), hipMemcpyDeviceToHost, st));
  HIPC(hipStreamSynchronize(st));
  r->n_compute = reinterpret_cast<const DecideOut*>(r->dec_host)->n_compute;
  const uint8_t* mk = r->mask_h();
  for (int s = 0; s < r->S; ++s) if (mk[s]) r->has_ref_h[s] = 1;
  if (mask_out) memcpy(mask_out, mk, r->S);
  if (a_out) memcpy(a_out, r->a_seen_h(), r->S * sizeof(double));
  r->decided_step = step;
  return CS_OK;
}

cs_status cs_cache_decide(cs_rollout* r, int32_t step, const uint8_t* ovr, uint8_t* mask_out,
                          double* a_out) {
  GUARD({ return decide_impl(r, step, ovr, mask_out, a_out); })
}

static cs_status step_impl(cs_rollout* r, int32_t step) {
  CHECK(r, CS_E_INVAL, "rollout is NULL");
  CHECK(step >= 1 && step <= r->desc.n_steps, CS_E_INVAL, "step %d outside 1..%d", step, r->desc.n_steps);
  CHECK(step == r->steps_done + 1, CS_E_STATE, "step %d requested, next step is %d", step, r->steps_done + 1);
  if (r->decided_step != step) TRY(decide_impl(r, step, nullptr, nullptr, nullptr));
  cs_model* m = r->model;
  hipStream_t st = m->stream;
  const cs_rollout_desc& d = r->desc;
  // the decision kernel left the computed streams (and their text branch)
  // compacted on the device; only their count was read back
  if (d.mode == CS_CACHE_PAB) {
    // every call computes (the decision compacted all S streams in order);
    // the attention branches follow the broadcast schedule
    CHECK(r->n_compute == r->S, CS_E_STATE, "PAB step %d: %d of %d calls computing", step,
          r->n_compute, r->S);
    const bool window = step <= d.k_warm || step > d.n_steps - d.k_cool;
    const bool cs_ = window || !r->pab_have_self || (step - d.k_warm) % d.pab_self_range == 0;
    const bool cc_ = window || !r->pab_have_cross || (step - d.k_warm) % d.pab_cross_range == 0;
    PabIO io{r->pab_self, r->pab_cross, cs_ ? PAB_STORE : PAB_REUSE, cc_ ? PAB_STORE : PAB_REUSE};
    TRY(dit_dispatch(m, r->ws, r->ctx, r->x, r->slots, r->branch, r->n_compute, d.n_branch,
                     r->t[step - 1], r->vbuf, &io));
    r->pab_have_self = r->pab_have_cross = true;
    if (!cs_) r->self_reused += r->S;
    if (!cc_) r->cross_reused += r->S;
  } else if (r->n_compute > 0) {
    TRY(dit_dispatch(m, r->ws, r->ctx, r->x, r->slots, r->branch, r->n_compute, d.n_branch,
                     r->t[step - 1], r->vbuf));
  }
  {
    ProfScope ps(m->prof, CS_K_UPDATE, st);
    const float dt = r->t[step] - r->t[step - 1];
    const int store_state = d.mode == CS_CACHE_ADAPTIVE || d.mode == CS_CACHE_STATIC;
    HIPC(cache_update(r->x, r->xref, r->delta, r->vbuf, r->mask_dev(), d.n_cand, d.n_branch, r->D, dt,
                      d.guidance, store_state, r->vtil, st));
    if (r->vtil) r->vtil_step = step;
  }
  r->calls += r->S;
  r->computed += r->n_compute;
  r->steps_done = step;
  return CS_OK;
}

cs_status cs_denoise_step(cs_rollout* r, int32_t step) { GUARD({ return step_impl(r, step); }) }

cs_status cs_score(cs_rollout* r, const float* w, double* scores) {
  GUARD({
    CHECK(r, CS_E_INVAL, "rollout is NULL");
    CHECK(w && scores, CS_E_INVAL, "w and scores must be non-NULL");
    cs_model* m = r->model;
    hipStream_t st = m->stream;
    {
      ProfScope ps(m->prof, CS_K_SCORE, st);
      HIPC(score_partials(r->x, nullptr, 0.0f, w, r->desc.n_cand, r->D, r->spart, st));
      HIPC(score_finalize(r->spart, r->desc.n_cand, r->nschunk, r->D, r->scores, st));
    }
    HIPC(hipMemcpyAsync(r->scores_host, r->scores, r->desc.n_cand * sizeof(double), hipMemcpyDeviceToHost, st));
    HIPC(hipStreamSynchronize(st));
    memcpy(scores, r->scores_host, r->desc.n_cand * sizeof(double));
    return CS_OK;
  })
}

cs_status cs_score_noalloc(const float* x, const float* w, int32_t n, int64_t D, double* scores,
                           void* stream) {
  GUARD({
    CHECK(x && w && scores, CS_E_INVAL, "x, w and scores must be non-NULL");
    CHECK(n >= 1 && n <= 65535, CS_E_INVAL, "n must be in [1, 65535]");
    CHECK(D >= 4 && D % 4 == 0, CS_E_INVAL, "D must be a positive multiple of 4");
    CHECK(((uintptr_t)x % 16) == 0 && ((uintptr_t)w % 16) == 0, CS_E_INVAL,
          "x and w must be 16-byte aligned");
    CHECK(((uintptr_t)scores % 8) == 0, CS_E_INVAL, "scores must be 8-byte aligned");
    const long nchunk = score_chunks((long)D);
    CHECK((long)n * nchunk <= (long)CS_SCORE_NOALLOC_MAX_PARTIALS, CS_E_INVAL,
          "n * ceil(D / 8192) = %ld partial sums exceed the scratch capacity of %ld", (long)n * nchunk,
          (long)CS_SCORE_NOALLOC_MAX_PARTIALS);
    double* part = nullptr;
    TRY(scratch_ptr(&part));
    hipStream_t st = (hipStream_t)stream;
    // every partial the finalize reads is written by the partials kernel of
    // this call first (same stream), so the array needs no clearing
    HIPC(score_partials(x, nullptr, 0.0f, w, n, (long)D, part, st));
    HIPC(score_finalize(part, n, (int)nchunk, (long)D, scores, st));
    return CS_OK;
  })
}

cs_status cs_rollout_enable_preview(cs_rollout* r, int32_t on) {
  GUARD({
    CHECK(r, CS_E_INVAL, "rollout is NULL");
    if (on && !r->vtil) {
      TRY(dmalloc((void**)&r->vtil, (size_t)r->desc.n_cand * r->D * sizeof(float)));
      r->vtil_step = -1;
    } else if (!on && r->vtil) {
      HIPC(hipStreamSynchronize(r->model->stream));
      HIPC(hipFree(r->vtil));
      r->vtil = nullptr;
      r->vtil_step = -1;
    }
    return CS_OK;
  })
}

cs_status cs_preview_score(cs_rollout* r, const float* w, double* scores) {
  GUARD({
    CHECK(r, CS_E_INVAL, "rollout is NULL");
    CHECK(w && scores, CS_E_INVAL, "w and scores must be non-NULL");
    CHECK(r->vtil && r->vtil_step == r->steps_done && r->steps_done >= 1, CS_E_STATE,
          "preview needs cs_rollout_enable_preview before the last completed step");
    cs_model* m = r->model;
    hipStream_t st = m->stream;
    const float t_next = r->t[r->steps_done];
    {
      ProfScope ps(m->prof, CS_K_SCORE, st);
      HIPC(score_partials(r->x, r->vtil, t_next, w, r->desc.n_cand, r->D, r->spart, st));
      HIPC(score_finalize(r->spart, r->desc.n_cand, r->nschunk, r->D, r->scores, st));
    }
    HIPC(hipMemcpyAsync(r->scores_host, r->scores, r->desc.n_cand * sizeof(double), hipMemcpyDeviceToHost, st));
    HIPC(hipStreamSynchronize(st));
    memcpy(scores, r->scores_host, r->desc.n_cand * sizeof(double));
    return CS_OK;
  })
}

cs_status cs_rollout_retain(cs_rollout* r, const int32_t* keep, int32_t n_keep) {
  GUARD({
    CHECK(r && keep, CS_E_INVAL, "rollout and keep must be non-NULL");
    CHECK(r->desc.mode != CS_CACHE_PAB, CS_E_UNSUPPORTED, "retain is not available in CS_CACHE_PAB mode");
    const int N = r->desc.n_cand, B = r->desc.n_branch;
    CHECK(n_keep >= 1 && n_keep <= N, CS_E_INVAL, "n_keep must be in [1, %d]", N);
    for (int j = 0; j < n_keep; ++j) {
      CHECK(keep[j] >= 0 && keep[j] < N, CS_E_INVAL, "keep[%d] = %d out of range", j, keep[j]);
      CHECK(j == 0 || keep[j] > keep[j - 1], CS_E_INVAL, "keep must be strictly increasing");
    }
    CHECK(r->decided_step != r->steps_done + 1, CS_E_STATE,
          "retain between cs_cache_decide and cs_denoise_step is not supported");
    hipStream_t st = r->model->stream;
    const size_t D = r->D;
    // keep[j] >= j, so copying in increasing j never overwrites a source
    // that a later copy still needs; the copies are ordered on the stream.
    for (int j = 0; j < n_keep; ++j) {
      const int i = keep[j];
      if (i == j) continue;
      HIPC(hipMemcpyAsync(r->x + j * D, r->x + i * D, D * 4, hipMemcpyDeviceToDevice, st));
      if (r->vtil) HIPC(hipMemcpyAsync(r->vtil + j * D, r->vtil + i * D, D * 4, hipMemcpyDeviceToDevice, st));
      HIPC(hipMemcpyAsync(r->xref + (size_t)j * B * D, r->xref + (size_t)i * B * D, B * D * 4,
                          hipMemcpyDeviceToDevice, st));
      HIPC(hipMemcpyAsync(r->delta + (size_t)j * B * D, r->delta + (size_t)i * B * D, B * D * 4,
                          hipMemcpyDeviceToDevice, st));
      HIPC(hipMemcpyAsync(r->a + (size_t)j * B, r->a + (size_t)i * B, B * sizeof(double),
                          hipMemcpyDeviceToDevice, st));
      HIPC(hipMemcpyAsync(r->has_ref + (size_t)j * B, r->has_ref + (size_t)i * B, B,
                          hipMemcpyDeviceToDevice, st));
      for (int b = 0; b < B; ++b) r->has_ref_h[j * B + b] = r->has_ref_h[i * B + b];
    }
    HIPC(hipStreamSynchronize(st));
    r->desc.n_cand = n_keep;
    r->S = n_keep * B;
    r->has_ref_h.resize(r->S);
    r->decided_step = 0;
    return CS_OK;
  })
}

cs_status cs_rollout_latents(cs_rollout* r, float* dst) {
  GUARD({
    CHECK(r && dst, CS_E_INVAL, "rollout and dst must be non-NULL");
    HIPC(hipMemcpyAsync(dst, r->x, (size_t)r->desc.n_cand * r->D * sizeof(float), hipMemcpyDeviceToDevice,
                        r->model->stream));
    return CS_OK;
  })
}

cs_status cs_rollout_stats(cs_rollout* r, cs_rollout_stats_t* out) {
  GUARD({
    CHECK(r && out, CS_E_INVAL, "rollout and out must be non-NULL");
    out->steps_done = r->steps_done;
    out->calls = r->calls;
    out->computed = r->computed;
    out->self_reused = r->self_reused;
    out->cross_reused = r->cross_reused;
    out->n_cand = r->desc.n_cand;
    return CS_OK;
  })
}

// checkpoint layout: header | x | xref | delta | a | has_ref
struct CkptHeader { uint64_t magic; int32_t n_cand, n_branch, steps_done, pad; int64_t D; };
static const uint64_t CKPT_MAGIC = 0x43535f524f4c4c31ull;  // "CS_ROLL1"

cs_status cs_rollout_export(cs_rollout* r, void* buf, size_t* bytes) {
  GUARD({
    CHECK(r && bytes, CS_E_INVAL, "rollout and bytes must be non-NULL");
    CHECK(r->desc.mode != CS_CACHE_PAB, CS_E_UNSUPPORTED, "checkpoints are not available in CS_CACHE_PAB mode");
    const size_t N = r->desc.n_cand, S = r->S, D = r->D;
    const size_t need = sizeof(CkptHeader) + (N * D + 2 * S * D) * sizeof(float) + S * sizeof(double) + S;
    if (!buf) { *bytes = need; return CS_OK; }
    CHECK(*bytes >= need, CS_E_INVAL, "buffer holds %zu bytes, %zu needed", *bytes, need);
    CHECK(r->decided_step != r->steps_done + 1 || r->steps_done == r->desc.n_steps, CS_E_STATE,
          "export between cs_cache_decide and cs_denoise_step is not supported");
    hipStream_t st = r->model->stream;
    char* p = (char*)buf;
    CkptHeader h{CKPT_MAGIC, r->desc.n_cand, r->desc.n_branch, r->steps_done, 0, (int64_t)D};
    memcpy(p, &h, sizeof(h));
    p += sizeof(h);
    HIPC(hipMemcpyAsync(p, r->x, N * D * 4, hipMemcpyDeviceToHost, st)); p += N * D * 4;
    HIPC(hipMemcpyAsync(p, r->xref, S * D * 4, hipMemcpyDeviceToHost, st)); p += S * D * 4;
    HIPC(hipMemcpyAsync(p, r->delta, S * D * 4, hipMemcpyDeviceToHost, st)); p += S * D * 4;
    HIPC(hipMemcpyAsync(p, r->a, S * 8, hipMemcpyDeviceToHost, st)); p += S * 8;
    HIPC(hipMemcpyAsync(p, r->has_ref, S, hipMemcpyDeviceToHost, st));
    HIPC(hipStreamSynchronize(st));
    *bytes = need;
    return CS_OK;
  })
}

cs_status cs_rollout_import(cs_rollout* r, const void* buf, size_t bytes) {
  GUARD({
    CHECK(r && buf, CS_E_INVAL, "rollout and buf must be non-NULL");
    CHECK(r->desc.mode != CS_CACHE_PAB, CS_E_UNSUPPORTED, "checkpoints are not available in CS_CACHE_PAB mode");
    const size_t N = r->desc.n_cand, S = r->S, D = r->D;
    const size_t need = sizeof(CkptHeader) + (N * D + 2 * S * D) * sizeof(float) + S * sizeof(double) + S;
    CHECK(bytes == need, CS_E_INVAL, "checkpoint has %zu bytes, %zu expected", bytes, need);
    CkptHeader h;
    memcpy(&h, buf, sizeof(h));
    CHECK(h.magic == CKPT_MAGIC && h.n_cand == r->desc.n_cand && h.n_branch == r->desc.n_branch &&
              h.D == (int64_t)D && h.steps_done >= 0 && h.steps_done <= r->desc.n_steps,
          CS_E_INVAL, "checkpoint does not match this rollout");
    hipStream_t st = r->model->stream;
    const char* p = (const char*)buf + sizeof(h);
    HIPC(hipMemcpyAsync(r->x, p, N * D * 4, hipMemcpyHostToDevice, st)); p += N * D * 4;
    HIPC(hipMemcpyAsync(r->xref, p, S * D * 4, hipMemcpyHostToDevice, st)); p += S * D * 4;
    HIPC(hipMemcpyAsync(r->delta, p, S * D * 4, hipMemcpyHostToDevice, st)); p += S * D * 4;
    HIPC(hipMemcpyAsync(r->a, p, S * 8, hipMemcpyHostToDevice, st)); p += S * 8;
    HIPC(hipMemcpyAsync(r->has_ref, p, S, hipMemcpyHostToDevice, st));
    HIPC(hipStreamSynchronize(st));
    r->has_ref_h.assign((const uint8_t*)p, (const uint8_t*)p + S);
    r->steps_done = h.steps_done;
    r->decided_step = 0;
    return CS_OK;
  })
}

// ------------------------------------------------------------------ ranking
cs_status cs_rank(const double* sc, const double* sf, int32_t n, int32_t* order_c, int32_t* order_f,
                  double* rho, int32_t* top1) {
  GUARD({
    CHECK(sc, CS_E_INVAL, "s_cached must be non-NULL");
    if (!sf) {
      CHECK(n >= 1, CS_E_INVAL, "n must be >= 1");
      CHECK(!order_f && !rho && !top1, CS_E_INVAL,
            "order_full, rho and top1_agree need s_full; pass NULL for them");
    } else {
      CHECK(n >= 2, CS_E_INVAL, "n must be >= 2");
    }
    for (int i = 0; i < n; ++i)
      CHECK(!(sc[i] != sc[i]) && !(sf && sf[i] != sf[i]), CS_E_INVAL, "scores must not be NaN");
    auto order = [n](const double* s) {
      std::vector<int32_t> o(n);
      for (int i = 0; i < n; ++i) o[i] = i;
      std::stable_sort(o.begin(), o.end(), [s](int32_t a, int32_t b) { return s[a] > s[b]; });
      return o;
    };
    auto ranks = [n](const double* s) {
      std::vector<int32_t> o(n);
      for (int i = 0; i < n; ++i) o[i] = i;
      std::stable_sort(o.begin(), o.end(), [s](int32_t a, int32_t b) { return s[a] < s[b]; });
      std::vector<double> r(n);
      int i = 0;
      while (i < n) {
        int j = i;
        while (j + 1 < n && s[o[j + 1]] == s[o[i]]) ++j;
        const double avg = 0.5 * (i + j) + 1.0;
        for (int k = i; k <= j; ++k) r[o[k]] = avg;
        i = j + 1;
      }
      return r;
    };
    const std::vector<int32_t> oc = order(sc);
    if (order_c) memcpy(order_c, oc.data(), n * sizeof(int32_t));
    if (!sf) return CS_OK;
    const std::vector<int32_t> of = order(sf);
    if (order_f) memcpy(order_f, of.data(), n * sizeof(int32_t));
    if (top1) *top1 = oc[0] == of[0] ? 1 : 0;
    if (rho) {
      const std::vector<double> rc = ranks(sc), rf = ranks(sf);
      double mc = 0, mf = 0;
      for (int i = 0; i < n; ++i) { mc += rc[i]; mf += rf[i]; }
      mc /= n;
      mf /= n;
      double sxy = 0, sxx = 0, syy = 0;
      for (int i = 0; i < n; ++i) {
        sxy += (rc[i] - mc) * (rf[i] - mf);
        sxx += (rc[i] - mc) * (rc[i] - mc);
        syy += (rf[i] - mf) * (rf[i] - mf);
      }
      *rho = (sxx == 0.0 || syy == 0.0) ? NAN : sxy / sqrt(sxx * syy);
    }
    return CS_OK;
  })
}

// ----------------------------------------------------------------- profiler
cs_status cs_profile_enable(cs_model* m, int32_t on) {
  GUARD({
    CHECK(m, CS_E_INVAL, "model is NULL");
    m->prof.on = on != 0;
    return CS_OK;
  })
}

cs_status cs_profile_reset(cs_model* m) {
  GUARD({
    CHECK(m, CS_E_INVAL, "model is NULL");
    HIPC(hipStreamSynchronize(m->stream));
    m->prof.reset();
    return CS_OK;
  })
}

cs_status cs_profile_read(cs_model* m, int32_t fam, double* total_ms, int64_t* launches) {
  GUARD({
    CHECK(m, CS_E_INVAL, "model is NULL");
    CHECK(fam >= 0 && fam < CS_K_COUNT, CS_E_INVAL, "unknown kernel family %d", fam);
    HIPC(hipStreamSynchronize(m->stream));
    m->prof.flush();
    if (total_ms) *total_ms = m->prof.total[fam];
    if (launches) *launches = m->prof.count[fam];
    return CS_OK;
  })
}

}  // extern "C"
