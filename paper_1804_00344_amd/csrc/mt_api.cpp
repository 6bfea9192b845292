// libmtstep C ABI: argument validation, weight packing, workspace layout and the launch
// sequence of one decoder step (declarations and contracts in include/mtstep.h).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "mt_internal.h"

using namespace mt;

namespace {

thread_local char g_err[512] = "";

mt_status fail(mt_status s, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return s;
}

#define HIP_TRY(expr)                                                                      \
  do {                                                                                     \
    hipError_t e_ = (expr);                                                                \
    if (e_ != hipSuccess) return fail(MT_ERR_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

constexpr uint32_t kMagic = 0x4d545350u;  // "MTSP"
constexpr int kNPad = 256;                // N padding of packed weights (>= any tile BN)
constexpr int kKPad = 64;                 // K padding of fp32 weights (a multiple of 4 k-steps)
constexpr int kKPadFrag = 128;            // K padding of bf16 weights (one LDS stage)
// Row counts the products are expected to run at, for the choice of the fp32 fragment form
// (64 sentences x beam 12, their 5000 or so source positions, the sentences): a model serves
// any batch, only the speed of other row counts may differ.
constexpr long kRefRows = 768, kRefCtxRows = 4096, kRefSentences = 64;
constexpr int kMaxTransitions = 16;  // recurrent-only GRU blocks after GRU 2

size_t rup(size_t x, size_t a) { return (x + a - 1) / a * a; }

struct Packed {
  void *p = nullptr;
  int N = 0, K = 0, ldb = 0;
  int blk = 16;  // fp32: column block width of the fragment order (16 or 32)
};

struct ProfSlot {
  std::vector<std::pair<hipEvent_t, hipEvent_t>> pending;
  double ms = 0.0;
  int64_t n = 0;
  uint64_t seen = 0;  // launches of the class since the last reset (timed or not)
};

}  // namespace

struct mt_model {
  uint32_t magic;
  mt_config cfg;
  int C;
  int bf16;       // gemm dtype is bf16
  int esize;      // bytes per GEMM operand element
  Packed w1x, w1h, w2, w3, w4, wp, ws0;  // packed [N_pad][K_pad]
  void *wo_frag;  // output matrix in MFMA fragment order (vocabulary kernel)
  Packed wsamp;   // its first vocab_sample_size(V) columns in the GEMM layout (threshold pass)
  float *bo_pad;  // output bias padded to a multiple of kVocabPad with -inf
  int logit_bounded;  // every logit provably in [-40, 40] (see mt_load_weights)
  int num_cu;
  void *emb;      // [V][E] fp32
  float *embx;    // [V][3H+E] fp32: emb [W1 | Wt_y] + [b1 | 0], the token side of GRU 1 and the readout
  float *bias1x, *bias3, *ba, *bi, *bt, *va;
  float *ln[10];  // g1a be1a g1u be1u g2a be2a g2u be2u gt bet
  Packed wp2;                     // dual-source models: second source's key projection Ua2
  float *ba2 = nullptr, *va2 = nullptr;
  Packed wenc_x, wenc_f, wenc_b;  // encoder: [Wef | Web], Uef, Ueb
  float *bias_enc = nullptr;      // [bef | beb]
  float *semb = nullptr;          // [src_V][E] fp32 source embeddings
  std::vector<Packed> wenc_tf, wenc_tb;  // encoder transition blocks, per block and direction
  float *bias_tenc = nullptr;            // [block][direction][3H]
  // encoder layer norm: input-block gains/shifts of both paths [direction][3H] (gea, bea,
  // geu, beu), transition blocks' recurrent-path gains/shifts [direction][block][3H]
  float *ln_enc[6] = {nullptr, nullptr, nullptr, nullptr, nullptr, nullptr};
  std::vector<Packed> wtr;        // transition blocks' recurrent matrices
  float *btr = nullptr;           // [T][3H] their biases
  float *gtu = nullptr, *betu = nullptr;  // [T][3H] layer norm of their recurrent products
  int device;     // the HIP device the model was loaded on
  // sentence order (longest first) of each source's attention, written by the precompute of
  // a batch of srank_B[i] sentences (-1: none yet); it only schedules the attention rows
  int *srank[2] = {nullptr, nullptr};
  int srank_B[2] = {-1, -1};
  int32_t *err;
  unsigned long long *nrecompute;  // rows whose fused candidates were recomputed exactly
  std::vector<void *> allocs;
  // call-order state for mt_beam_topk(logp = NULL)
  int last_B = -1, last_K = -1;
  const void *last_ws = nullptr;
  int last_ens_n = 0;      // the last step ran as the last of this many fused-ensemble members (0: not)
  float last_ens_w = 0.f;  // and with this weight
  int last_ens_joint = 0;  // the last step was a member of this many for the joint vocabulary pass
  // bf16 copy of a state the step wrote (mt_set_state_reuse): state_out, workspace and rows of
  // the last step, whose workspace holds the copy (cleared by every other call on the model)
  int reuse_state = 0;
  const void *shadow_of = nullptr, *shadow_ws = nullptr;
  int shadow_rows = 0;
  // profiling
  uint32_t prof_mask = 0;
  uint32_t prof_every = 1;  // time one launch in this many of each selected class
  ProfSlot prof[MT_KERNEL_COUNT];
  std::vector<hipEvent_t> ev_pool;
};

namespace {

bool valid_model(const mt_model *m) { return m && m->magic == kMagic; }

bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

mt_status check_cfg(const mt_config *c) {
  if (!c) return fail(MT_ERR_ARG, "config is NULL");
  auto dim_ok = [](int v, int lo, int hi) { return v >= lo && v <= hi && v % 16 == 0; };
  if (!dim_ok(c->E, 16, 4096)) return fail(MT_ERR_SHAPE, "E=%d: need a multiple of 16 in [16, 4096]", c->E);
  if (!dim_ok(c->H, 16, 4096)) return fail(MT_ERR_SHAPE, "H=%d: need a multiple of 16 in [16, 4096]", c->H);
  if (!dim_ok(c->A, 16, 4096)) return fail(MT_ERR_SHAPE, "A=%d: need a multiple of 16 in [16, 4096]", c->A);
  if (c->V < 2 || c->V > (1 << 24)) return fail(MT_ERR_SHAPE, "V=%d: need 2 <= V <= 2^24", c->V);
  if (c->k_max < 1 || c->k_max > kKMax) return fail(MT_ERR_SHAPE, "k_max=%d: need 1..%d", c->k_max, kKMax);
  if (c->k_max > c->V) return fail(MT_ERR_SHAPE, "k_max=%d exceeds V=%d", c->k_max, c->V);
  if (c->layer_norm != 0 && c->layer_norm != 1) return fail(MT_ERR_ARG, "layer_norm must be 0 or 1");
  if (c->tied_output != 0 && c->tied_output != 1) return fail(MT_ERR_ARG, "tied_output must be 0 or 1");
  if (c->gemm_dtype != MT_F32 && c->gemm_dtype != MT_BF16)
    return fail(MT_ERR_DTYPE, "gemm_dtype=%d: need MT_F32 or MT_BF16", c->gemm_dtype);
  if (c->dual_source != 0 && c->dual_source != 1) return fail(MT_ERR_ARG, "dual_source must be 0 or 1");
  if (c->src_V < 0 || c->src_V > (1 << 24)) return fail(MT_ERR_SHAPE, "src_V=%d: need 0 <= src_V <= 2^24", c->src_V);
  if (c->dec_transitions < 0 || c->dec_transitions > kMaxTransitions)
    return fail(MT_ERR_SHAPE, "dec_transitions=%d: need 0..%d", c->dec_transitions, kMaxTransitions);
  if (c->enc_transitions < 0 || c->enc_transitions > kMaxTransitions)
    return fail(MT_ERR_SHAPE, "enc_transitions=%d: need 0..%d", c->enc_transitions, kMaxTransitions);
  if (c->enc_transitions > 0 && c->src_V <= 0)
    return fail(MT_ERR_ARG, "enc_transitions=%d needs an encoder (src_V > 0)", c->enc_transitions);
  if (c->enc_layer_norm != 0 && c->enc_layer_norm != 1) return fail(MT_ERR_ARG, "enc_layer_norm must be 0 or 1");
  if (c->enc_layer_norm && c->src_V <= 0) return fail(MT_ERR_ARG, "enc_layer_norm needs an encoder (src_V > 0)");
  if ((c->layer_norm || c->enc_layer_norm) && !(c->ln_eps > 0.f && std::isfinite(c->ln_eps)))
    return fail(MT_ERR_ARG, "ln_eps must be positive and finite");
  if (vocab_rows_per_block(c->gemm_dtype == MT_BF16, c->E) == 0)
    return fail(MT_ERR_SHAPE, "E=%d too large for the vocabulary kernel (E <= %d)", c->E,
                c->gemm_dtype == MT_BF16 ? 2048 : 1024);
  return MT_OK;
}

uint16_t bf16_bits(float f) { return bf16_rne_bits(f); }

struct Seg {
  const float *w;  // logical [K][ncols] row-major
  int ncols;
};

// W = concat(segments) [K][N], zero padded to [rup(K, kKPad or kKPadFrag)][rup(N, kNPad)], in the
// MFMA fragment order of the GEMM kernels: 16 bytes per lane l of each (column block nb, k-step
// ks) at ((nb * KS + ks) * 64 + l) * 16, KS = K_pad / (k per step):
//  fp32, 16-column blocks, 16-k steps: lane l holds column nb*16 + l%16, k = ks*16 + (l/16)*4 + 0..3;
//  fp32, 32-column blocks, 8-k steps:  lane l holds column nb*32 + l%32, k = ks*8 + (l/32)*4 + 0..3;
//  bf16, 32-column blocks, 16-k steps: lane l holds column nb*32 + l%32, k = ks*16 + (l/32)*8 + 0..7.
std::vector<char> pack_host(const std::vector<Seg> &segs, int K, int esize, int blk, int *N_out, int *ldb_out) {
  int N = 0;
  for (auto &s : segs) N += s.ncols;
  const int Np = (int)rup(N, kNPad), Kp = (int)rup(K, esize == 2 ? kKPadFrag : kKPad);
  std::vector<char> buf((size_t)Np * Kp * esize, 0);
  int n0 = 0;
  for (auto &s : segs) {
    for (int kb = 0; kb < K; kb += 64)
      for (int nb = 0; nb < s.ncols; nb += 64)
        for (int k = kb; k < std::min(K, kb + 64); ++k) {
          const float *src = s.w + (size_t)k * s.ncols;
          for (int n = nb; n < std::min(s.ncols, nb + 64); ++n) {
            const int nn = n0 + n;
            if (esize == 4 && blk == 32) {
              const int lane = (nn & 31) + 32 * ((k & 7) >> 2);
              const size_t o = ((((size_t)(nn >> 5) * (Kp / 8) + (k >> 3)) * 64 + lane) * 4) + (k & 3);
              ((float *)buf.data())[o] = src[n];
            } else if (esize == 4) {
              const int lane = (nn & 15) + 16 * ((k & 15) >> 2);
              const size_t o = ((((size_t)(nn >> 4) * (Kp / 16) + (k >> 4)) * 64 + lane) * 4) + (k & 3);
              ((float *)buf.data())[o] = src[n];
            } else {
              const int lane = (nn & 31) + 32 * ((k & 15) >> 3);
              const size_t o = ((((size_t)(nn >> 5) * (Kp / 16) + (k >> 4)) * 64 + lane) * 8) + (k & 7);
              ((uint16_t *)buf.data())[o] = bf16_bits(src[n]);
            }
          }
        }
    n0 += s.ncols;
  }
  *N_out = N;
  *ldb_out = Kp;
  return buf;
}

mt_status dev_upload(mt_model *m, const void *host, size_t bytes, void **out) {
  void *d = nullptr;
  const hipError_t e = hipMalloc(&d, bytes ? bytes : 16);
  if (e != hipSuccess) return fail(MT_ERR_OOM, "hipMalloc(%zu): %s", bytes, hipGetErrorString(e));
  m->allocs.push_back(d);
  if (bytes && host) HIP_TRY(hipMemcpy(d, host, bytes, hipMemcpyHostToDevice));
  *out = d;
  return MT_OK;
}

// rows: the row count the product is expected to run at (it picks the fp32 fragment form; any
// row count computes the same product)
mt_status upload_packed(mt_model *m, const std::vector<Seg> &segs, int K, long rows, Packed *p) {
  int N = 0;
  for (auto &s : segs) N += s.ncols;
  const int blk = m->esize == 4 ? gemm_f32_weight_block(rows, N, K) : 32;
  int ldb = 0;
  std::vector<char> buf = pack_host(segs, K, m->esize, blk, &N, &ldb);
  p->N = N;
  p->K = K;
  p->ldb = ldb;
  p->blk = blk;
  return dev_upload(m, buf.data(), buf.size(), &p->p);
}

mt_status upload_vec(mt_model *m, const std::vector<float> &v, float **out) {
  return dev_upload(m, v.data(), v.size() * sizeof(float), (void **)out);
}

std::vector<float> cat(std::initializer_list<std::pair<const float *, int>> parts) {
  std::vector<float> v;
  for (auto &p : parts) {
    if (p.first)
      v.insert(v.end(), p.first, p.first + p.second);
    else
      v.insert(v.end(), (size_t)p.second, 0.f);
  }
  return v;
}

// ---- workspace ----
struct WsLayout {
  size_t gh, s1, g2, c, g3, g4, t, sample, thr, part, cbuf, ccnt, lse, rowc, scand, scnt, s1h, ch, sth, sx, total;
  int ntiles, kc, nchunks;
};

WsLayout ws_layout(const mt_model *m, int B, int K) {
  const mt_config &c = m->cfg;
  const size_t M = (size_t)B * K, E = c.E, H = c.H, A = c.A, C = 2 * H;
  WsLayout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += rup(bytes, 256);
    return o;
  };
  L.gh = take(M * 3 * H * 4);
  L.s1 = take(M * H * 4);
  const size_t nsrc = m->cfg.dual_source ? 2 : 1;  // attention queries / contexts per row
  L.g2 = take(M * (nsrc * A + 3 * H) * 4);
  L.c = take(M * nsrc * C * 4);
  L.g3 = take(M * (3 * H + E) * 4);
  L.g4 = take(M * E * 4);
  L.t = take(M * E * m->esize);
  L.ntiles = vocab_chunks(m->bf16, (int)M, c.V, c.E, m->num_cu);
  L.kc = K;
  L.sample = take(M * vocab_sample_size(c.V) * 4);
  L.thr = take(M * 4);
  L.part = take(M * L.ntiles * sizeof(float2));
  L.cbuf = take(M * L.ntiles * vocab_lists() * kVocabCap * sizeof(int2));
  L.ccnt = take(M * L.ntiles * vocab_lists() * sizeof(int));
  L.lse = take(M * 4);
  L.rowc = take(M * K * sizeof(int2));
  // chunks of a materialised row for the first selection level
  {
    int chunk = 0;
    topk_scan_shape((int)M, c.V, &chunk, &L.nchunks);
  }
  L.scand = take(M * L.nchunks * K * sizeof(int2));
  L.scnt = take((size_t)B * sizeof(int));
  // bf16 copies of s1, the context and the new state: the A operands of the bf16 products
  const size_t h16 = m->bf16 ? 2 : 0;
  L.s1h = take(M * H * h16);
  L.ch = take(M * nsrc * C * h16);
  L.sth = take(M * H * h16);
  // transition blocks alternate between state_out and this buffer
  L.sx = take(c.dec_transitions > 0 ? M * H * 4 : 0);
  L.total = off;
  return L;
}

// precompute workspace: masked means [B][2H] fp32, the valid-row list [B*S] and its count
static size_t rup256(size_t x) { return (x + 255) / 256 * 256; }
size_t precompute_ws_bytes(const mt_model *m, int B, int S) {
  return rup256((size_t)B * 2 * m->cfg.H * 4) + rup256((size_t)B * S * 4) + 256;
}

// Scratch of mt_precompute_ctx_noalloc: a file-scope device array, one copy per GPU, held
// until the process ends.  In host code `scratch` only names the symbol; its device address
// on each GPU comes from hipGetSymbolAddress with that GPU current, resolved once per device
// (at model load, or at the entry point's first call on a device) and kept in g_scratch.
constexpr size_t kNoAllocScratchBytes = size_t(16) << 20;
constexpr int kMaxDevices = 64;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];
std::mutex g_scratch_mu;
void *g_scratch[kMaxDevices] = {};

// device address of this device's scratch (dev must be the current device)
mt_status scratch_for_device(int dev, void **out) {
  if (dev < 0 || dev >= kMaxDevices) return fail(MT_ERR_HIP, "device %d out of range for the scratch table", dev);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch[dev]) {
    void *ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress((void **)&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
      return fail(MT_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
    g_scratch[dev] = ptr;
  }
  *out = g_scratch[dev];
  return MT_OK;
}

// ---- profiling ----
hipEvent_t get_event(mt_model *m) {
  if (!m->ev_pool.empty()) {
    hipEvent_t e = m->ev_pool.back();
    m->ev_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

void fold_profile(mt_model *m, int k) {
  ProfSlot &s = m->prof[k];
  for (auto &pr : s.pending) {
    float ms = 0.f;
    if (hipEventSynchronize(pr.second) == hipSuccess && hipEventElapsedTime(&ms, pr.first, pr.second) == hipSuccess) {
      s.ms += ms;
      s.n += 1;
    }
    m->ev_pool.push_back(pr.first);
    m->ev_pool.push_back(pr.second);
  }
  s.pending.clear();
}

struct Timed {  // records events around one launch when profiling is on
  mt_model *m;
  int k;
  hipStream_t st;
  hipEvent_t a = nullptr, b = nullptr;
  Timed(mt_model *m_, int k_, hipStream_t st_, bool on = true) : m(m_), k(k_), st(st_) {
    if (on && (m->prof_mask & (1u << k)) && m->prof[k].seen++ % m->prof_every == 0) {
      a = get_event(m);
      b = get_event(m);
      if (a && b) hipEventRecord(a, st);
    }
  }
  ~Timed() {
    if (a && b) {
      hipEventRecord(b, st);
      m->prof[k].pending.emplace_back(a, b);
      if (m->prof[k].pending.size() > 8192) fold_profile(m, k);
    }
  }
};

// LAUNCH_IF: timing events (when profiling selects the kernel class) only if `on`
#define LAUNCH_IF(kid, on, expr)                                                            \
  do {                                                                                      \
    hipError_t e_;                                                                          \
    {                                                                                       \
      Timed tm_(model, kid, st, on);                                                        \
      e_ = (expr);                                                                          \
    }                                                                                       \
    if (e_ != hipSuccess) return fail(MT_ERR_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)
#define LAUNCH(kid, expr) LAUNCH_IF(kid, true, expr)

mt_status check_dev_ptr(const void *p, const char *name, size_t align = 16) {
  if (!p) return fail(MT_ERR_ARG, "%s is NULL", name);
  if (!aligned(p, align)) return fail(MT_ERR_ARG, "%s is not %zu-byte aligned", name, align);
  return MT_OK;
}

#define CHECK(expr)                 \
  do {                              \
    mt_status s_ = (expr);          \
    if (s_ != MT_OK) return s_;     \
  } while (0)

}  // namespace

extern "C" {

const char *mt_last_error(void) { return g_err; }

void mt_round_bf16(const float *src, uint16_t *dst, size_t n) {
  if (!src || !dst) return;
  for (size_t i = 0; i < n; ++i) dst[i] = bf16_rne_bits(src[i]);
}

mt_status mt_load_weights(const mt_config *cfg, const mt_weights *w, mt_model **out) {
  g_err[0] = 0;
  if (!out) return fail(MT_ERR_ARG, "out is NULL");
  *out = nullptr;
  CHECK(check_cfg(cfg));
  if (!w) return fail(MT_ERR_ARG, "weights is NULL");
  const mt_config &c = *cfg;
  struct Need {
    const float *p;
    const char *n;
  } need[] = {{w->emb, "emb"}, {w->W1, "W1"}, {w->U1, "U1"}, {w->b1, "b1"}, {w->Ua, "Ua"},
              {w->ba, "ba"},   {w->Wa, "Wa"}, {w->va, "va"}, {w->W2, "W2"}, {w->U2, "U2"},
              {w->b2, "b2"},   {w->Wt_s, "Wt_s"}, {w->Wt_y, "Wt_y"}, {w->Wt_c, "Wt_c"},
              {w->bt, "bt"},   {w->bo, "bo"}, {w->Wi, "Wi"}, {w->bi, "bi"}};
  for (auto &n : need)
    if (!n.p) return fail(MT_ERR_ARG, "weight %s is NULL", n.n);
  if (!c.tied_output && !w->Wo) return fail(MT_ERR_ARG, "weight Wo is NULL (tied_output = 0)");
  const float *lnp[10] = {w->g1a, w->be1a, w->g1u, w->be1u, w->g2a, w->be2a, w->g2u, w->be2u, w->gt, w->bet};
  if (c.layer_norm)
    for (int i = 0; i < 10; ++i)
      if (!lnp[i]) return fail(MT_ERR_ARG, "layer-norm parameter %d is NULL (layer_norm = 1)", i);
  if (c.dual_source) {
    const float *dw[] = {w->Ua2, w->ba2, w->Wa2, w->va2};
    const char *dn[] = {"Ua2", "ba2", "Wa2", "va2"};
    for (int i = 0; i < 4; ++i)
      if (!dw[i]) return fail(MT_ERR_ARG, "second-source weight %s is NULL (dual_source = 1)", dn[i]);
  }
  if (c.src_V > 0) {
    const float *ew[] = {w->semb, w->Wef, w->Uef, w->bef, w->Web, w->Ueb, w->beb};
    const char *en[] = {"semb", "Wef", "Uef", "bef", "Web", "Ueb", "beb"};
    for (int i = 0; i < 7; ++i)
      if (!ew[i]) return fail(MT_ERR_ARG, "encoder weight %s is NULL (src_V = %d)", en[i], c.src_V);
    if (c.enc_transitions > 0 && (!w->Utef || !w->btef || !w->Uteb || !w->bteb))
      return fail(MT_ERR_ARG, "Utef, btef, Uteb or bteb is NULL (enc_transitions = %d)", c.enc_transitions);
    if (c.enc_layer_norm && (!w->gea || !w->bea || !w->geu || !w->beu))
      return fail(MT_ERR_ARG, "gea, bea, geu or beu is NULL (enc_layer_norm = 1)");
    if (c.enc_layer_norm && c.enc_transitions > 0 && (!w->gteu || !w->beteu))
      return fail(MT_ERR_ARG, "gteu or beteu is NULL (enc_layer_norm = 1, enc_transitions > 0)");
  }
  if (c.dec_transitions > 0) {
    if (!w->Ut || !w->btr) return fail(MT_ERR_ARG, "Ut or btr is NULL (dec_transitions = %d)", c.dec_transitions);
    if (c.layer_norm && (!w->gtu || !w->betu))
      return fail(MT_ERR_ARG, "gtu or betu is NULL (dec_transitions > 0, layer_norm = 1)");
  }

  mt_model *m = new (std::nothrow) mt_model();
  if (!m) return fail(MT_ERR_OOM, "host allocation failed");
  m->magic = kMagic;
  m->cfg = c;
  m->C = 2 * c.H;
  m->bf16 = c.gemm_dtype == MT_BF16;
  m->esize = m->bf16 ? 2 : 4;
  {
    int dev = 0, ncu = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || ncu <= 0) {
      delete m;
      return fail(MT_ERR_HIP, "cannot query the device's compute units");
    }
    m->num_cu = ncu;
    m->device = dev;
    void *sp = nullptr;  // this device's no-alloc scratch, resolved at set-up
    if (scratch_for_device(dev, &sp) != MT_OK) {
      char keep[sizeof g_err];
      std::memcpy(keep, g_err, sizeof keep);
      delete m;
      std::memcpy(g_err, keep, sizeof keep);
      return MT_ERR_HIP;
    }
  }
  const int E = c.E, H = c.H, A = c.A, V = c.V, C = 2 * c.H;
  mt_status s = MT_OK;
  auto run = [&]() -> mt_status {
    CHECK(upload_packed(m, {{w->W1, 3 * H}, {w->Wt_y, E}}, E, V, &m->w1x));
    CHECK(upload_packed(m, {{w->U1, 3 * H}}, H, kRefRows, &m->w1h));
    // dual-source models: s1 [Wa | Wa2 | U2], and the context product takes [c1 ; c2] (2C rows)
    if (c.dual_source)
      CHECK(upload_packed(m, {{w->Wa, A}, {w->Wa2, A}, {w->U2, 3 * H}}, H, kRefRows, &m->w2));
    else
      CHECK(upload_packed(m, {{w->Wa, A}, {w->U2, 3 * H}}, H, kRefRows, &m->w2));
    CHECK(upload_packed(m, {{w->W2, 3 * H}, {w->Wt_c, E}}, c.dual_source ? 2 * C : C, kRefRows, &m->w3));
    if (c.dual_source) {
      CHECK(upload_packed(m, {{w->Ua2, A}}, C, kRefCtxRows, &m->wp2));
      CHECK(upload_vec(m, cat({{w->ba2, A}}), &m->ba2));
      CHECK(upload_vec(m, cat({{w->va2, A}}), &m->va2));
    }
    CHECK(upload_packed(m, {{w->Wt_s, E}}, H, kRefRows, &m->w4));
    CHECK(upload_packed(m, {{w->Ua, A}}, C, kRefCtxRows, &m->wp));
    CHECK(upload_packed(m, {{w->Wi, H}}, C, kRefSentences, &m->ws0));
    {  // output layer: Wo^T rows (or emb rows when tied) in MFMA fragment order
      std::vector<char> buf(vocab_pack_bytes(m->bf16, V, E));
      vocab_pack_host(m->bf16, V, E, c.tied_output ? w->emb : w->Wo, c.tied_output, buf.data());
      CHECK(dev_upload(m, buf.data(), buf.size(), &m->wo_frag));
      const int S = vocab_sample_size(V);
      std::vector<float> ws((size_t)E * S, 0.f);  // [E][S]: the first S output columns
      for (int e = 0; e < E; ++e)
        for (int v = 0; v < S && v < V; ++v)
          ws[(size_t)e * S + v] = c.tied_output ? w->emb[(size_t)v * E + e] : w->Wo[(size_t)e * V + v];
      CHECK(upload_packed(m, {{ws.data(), S}}, E, kRefRows, &m->wsamp));
      std::vector<float> bp((V + kVocabPad - 1) / kVocabPad * kVocabPad, -INFINITY);
      std::copy(w->bo, w->bo + V, bp.begin());
      CHECK(upload_vec(m, bp, &m->bo_pad));
      // The readout activations are tanh outputs (|t_e| <= 1, also after bf16 rounding), so
      // |logit_v| <= sqrt(E) |Wo[:, v]|_2 + |bo_v| (Cauchy-Schwarz; the weights as the kernel
      // sees them, i.e. bf16-rounded for a bf16 model, plus a relative slack for rounding).
      // When that bound is at most 40 the vocabulary kernel sums exp(logit) with no running
      // maximum: no term can overflow (e^40 * V is far below the fp32 range) or underflow.
      std::vector<double> ss(V, 0.0);
      auto as_kernel_sees = [&](float x) {
        if (m->bf16) {
          const uint32_t hb = (uint32_t)bf16_bits(x) << 16;
          std::memcpy(&x, &hb, 4);
        }
        return (double)x;
      };
      if (c.tied_output) {
        for (int v = 0; v < V; ++v)
          for (int e = 0; e < E; ++e) {
            const double x = as_kernel_sees(w->emb[(size_t)v * E + e]);
            ss[v] += x * x;
          }
      } else {
        for (int e = 0; e < E; ++e)
          for (int v = 0; v < V; ++v) {
            const double x = as_kernel_sees(w->Wo[(size_t)e * V + v]);
            ss[v] += x * x;
          }
      }
      double bound = 0.0;
      for (int v = 0; v < V; ++v) {
        const double bv = std::sqrt((double)E * ss[v]) * 1.01 + std::fabs((double)w->bo[v]);
        if (!(bv <= bound)) bound = bv;  // NaN propagates as "unbounded"
      }
      m->logit_bounded = bound <= 40.0 ? 1 : 0;
    }
    // embedding rows stay fp32 (a bf16 model rounds them to bf16 when they are staged as the
    // GEMM operand, like every other fp32 activation)
    CHECK(dev_upload(m, w->emb, (size_t)V * E * sizeof(float), &m->emb));
    CHECK(upload_vec(m, cat({{w->b1, 3 * H}, {nullptr, E}}), &m->bias1x));
    CHECK(upload_vec(m, cat({{w->b2, 3 * H}, {nullptr, E}}), &m->bias3));
    CHECK(upload_vec(m, cat({{w->ba, A}}), &m->ba));
    CHECK(upload_vec(m, cat({{w->bi, H}}), &m->bi));
    CHECK(upload_vec(m, cat({{w->bt, E}}), &m->bt));
    CHECK(upload_vec(m, cat({{w->va, A}}), &m->va));
    for (int i = 0; i < 10; ++i) {
      m->ln[i] = nullptr;
      if (c.layer_norm) CHECK(upload_vec(m, cat({{lnp[i], i < 8 ? 3 * H : E}}), &m->ln[i]));
    }
    if (c.src_V > 0) {
      CHECK(upload_packed(m, {{w->Wef, 3 * H}, {w->Web, 3 * H}}, E, kRefCtxRows, &m->wenc_x));
      CHECK(upload_packed(m, {{w->Uef, 3 * H}}, H, kRefSentences, &m->wenc_f));
      CHECK(upload_packed(m, {{w->Ueb, 3 * H}}, H, kRefSentences, &m->wenc_b));
      CHECK(upload_vec(m, cat({{w->bef, 3 * H}, {w->beb, 3 * H}}), &m->bias_enc));
      CHECK(dev_upload(m, w->semb, (size_t)c.src_V * E * sizeof(float), (void **)&m->semb));
      const int Te = c.enc_transitions;
      m->wenc_tf.resize(Te);
      m->wenc_tb.resize(Te);
      std::vector<float> bte;
      for (int j = 0; j < Te; ++j) {
        const size_t o = (size_t)j * H * 3 * H;
        CHECK(upload_packed(m, {{w->Utef + o, 3 * H}}, H, kRefSentences, &m->wenc_tf[j]));
        CHECK(upload_packed(m, {{w->Uteb + o, 3 * H}}, H, kRefSentences, &m->wenc_tb[j]));
        bte.insert(bte.end(), w->btef + (size_t)j * 3 * H, w->btef + (size_t)(j + 1) * 3 * H);
        bte.insert(bte.end(), w->bteb + (size_t)j * 3 * H, w->bteb + (size_t)(j + 1) * 3 * H);
      }
      if (Te > 0) CHECK(upload_vec(m, bte, &m->bias_tenc));
      if (c.enc_layer_norm) {
        const float *src[4] = {w->gea, w->bea, w->geu, w->beu};
        for (int i = 0; i < 4; ++i) CHECK(upload_vec(m, cat({{src[i], 6 * H}}), &m->ln_enc[i]));
        if (Te > 0) {
          CHECK(upload_vec(m, cat({{w->gteu, 2 * Te * 3 * H}}), &m->ln_enc[4]));
          CHECK(upload_vec(m, cat({{w->beteu, 2 * Te * 3 * H}}), &m->ln_enc[5]));
        }
      }
    }
    const int T = c.dec_transitions;
    m->wtr.resize(T);
    for (int j = 0; j < T; ++j)
      CHECK(upload_packed(m, {{w->Ut + (size_t)j * H * 3 * H, 3 * H}}, H, kRefRows, &m->wtr[j]));
    if (T > 0) {
      CHECK(upload_vec(m, cat({{w->btr, T * 3 * H}}), &m->btr));
      if (c.layer_norm) {
        CHECK(upload_vec(m, cat({{w->gtu, T * 3 * H}}), &m->gtu));
        CHECK(upload_vec(m, cat({{w->betu, T * 3 * H}}), &m->betu));
      }
    }
    int32_t zero = 0;
    CHECK(dev_upload(m, &zero, sizeof zero, (void **)&m->err));
    unsigned long long zero64 = 0;
    CHECK(dev_upload(m, &zero64, sizeof zero64, (void **)&m->nrecompute));
    for (int i = 0; i < 2; ++i)
      CHECK(dev_upload(m, nullptr, (size_t)attention_order_max_sentences() * sizeof(int), (void **)&m->srank[i]));
    {
      // The token side of GRU 1 and of the readout, x [W1 | Wt_y] + [b1 | 0], depends only on
      // the token: it is computed once here for the whole vocabulary (same products, same
      // operand rounding as a per-step product) and the step gathers rows of it.
      CHECK(dev_upload(m, nullptr, (size_t)V * (3 * H + E) * sizeof(float), (void **)&m->embx));
      GemmProblem p{};
      p.A = m->emb; p.a_rows = V; p.lda = E; p.a_bf16 = 0;
      p.Bp = m->w1x.p; p.ldb = m->w1x.ldb; p.wblk = m->w1x.blk; p.bias = m->bias1x;
      p.out = m->embx; p.ldc = 3 * H + E; p.out_bf16 = 0;
      p.M = V; p.N = 3 * H + E; p.K = E;
      HIP_TRY(launch_gemm(m->bf16, &p, 1, EPI_STORE, nullptr));
      HIP_TRY(hipDeviceSynchronize());
    }
    return MT_OK;
  };
  s = run();
  if (s != MT_OK) {
    char keep[sizeof g_err];
    std::memcpy(keep, g_err, sizeof keep);
    mt_free(m);
    std::memcpy(g_err, keep, sizeof keep);
    return s;
  }
  *out = m;
  return MT_OK;
}

mt_status mt_free(mt_model *m) {
  if (!valid_model(m)) return fail(MT_ERR_ARG, "invalid model handle");
  hipDeviceSynchronize();
  for (int k = 0; k < MT_KERNEL_COUNT; ++k) {
    for (auto &pr : m->prof[k].pending) {
      hipEventDestroy(pr.first);
      hipEventDestroy(pr.second);
    }
  }
  for (auto e : m->ev_pool) hipEventDestroy(e);
  for (void *p : m->allocs) hipFree(p);
  m->magic = 0;
  delete m;
  return MT_OK;
}

size_t mt_workspace_bytes(const mt_model *m, int B, int K, int S) {
  if (!valid_model(m) || B < 1 || K < 1 || K > m->cfg.k_max || S < 1 || S > 1024) return 0;
  const WsLayout L = ws_layout(m, B, K);
  return std::max(L.total, precompute_ws_bytes(m, B, S));
}

// encoder workspace: input products [B*S][6H], recurrent products of both directions and a
// zero block [B][3H] each, fp32 states [2 directions][2][B][H] (bf16 models), intermediate
// states of the transition blocks [2 directions][B][H]
struct EncLayout {
  size_t xe, uf, ub, uz, st, tx, total;
};
static EncLayout enc_layout(const mt_model *m, int B, int S) {
  const size_t H = m->cfg.H;
  EncLayout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += rup256(bytes);
    return o;
  };
  L.xe = take((size_t)B * S * 6 * H * 4);
  L.uf = take((size_t)B * 3 * H * 4);
  L.ub = take((size_t)B * 3 * H * 4);
  L.uz = take((size_t)B * 3 * H * 4);
  L.st = take(m->bf16 ? (size_t)4 * B * H * 4 : 0);
  L.tx = take(m->cfg.enc_transitions > 0 ? (size_t)2 * B * H * 4 : 0);
  L.total = off;
  return L;
}

size_t mt_encode_workspace_bytes(const mt_model *m, int B, int S) {
  if (!valid_model(m) || m->cfg.src_V <= 0 || B < 1 || S < 1 || S > 1024 || (long long)B * S > (1 << 24)) return 0;
  return enc_layout(m, B, S).total;
}

mt_status mt_encode(mt_model *model, int B, int S, const int32_t *src_tok, const float *mask, void *ctx_out,
                    void *ws, size_t ws_bytes, void *stream) {
  g_err[0] = 0;
  if (!valid_model(model)) return fail(MT_ERR_ARG, "invalid model handle");
  model->shadow_of = nullptr;
  if (model->cfg.src_V <= 0) return fail(MT_ERR_STATE, "the model has no encoder (src_V = 0)");
  if (B < 1 || S < 1 || S > 1024) return fail(MT_ERR_SHAPE, "B=%d S=%d: need B >= 1, 1 <= S <= 1024", B, S);
  if ((long long)B * S > (1 << 24)) return fail(MT_ERR_SHAPE, "B*S exceeds 2^24");
  CHECK(check_dev_ptr(src_tok, "src_tok", 4));
  CHECK(check_dev_ptr(mask, "mask", 4));
  CHECK(check_dev_ptr(ctx_out, "ctx_out"));
  CHECK(check_dev_ptr(ws, "ws", 256));
  const EncLayout L = enc_layout(model, B, S);
  if (ws_bytes < L.total) return fail(MT_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, L.total);
  hipStream_t st = (hipStream_t)stream;
  const int H = model->cfg.H, E = model->cfg.E, C = 2 * H, bf = model->bf16;
  char *W = (char *)ws;
  float *xe = (float *)(W + L.xe), *uf = (float *)(W + L.uf), *ub = (float *)(W + L.ub), *uz = (float *)(W + L.uz);
  float *sst = (float *)(W + L.st);  // bf16 models: [dir][parity][B][H]
  const long ldc = (long)S * C;      // row stride of one sentence's positions in ctx_out
  // input side of every position and both directions: semb[src_tok] [Wef | Web] + [bef | beb]
  GemmProblem px{};
  px.A = model->semb; px.a_idx = src_tok; px.a_rows = model->cfg.src_V; px.lda = E; px.a_bf16 = 0;
  px.Bp = model->wenc_x.p; px.ldb = model->wenc_x.ldb; px.wblk = model->wenc_x.blk; px.bias = model->bias_enc;
  px.out = xe; px.ldc = 6 * H; px.M = B * S; px.N = 6 * H; px.K = E; px.err = model->err; px.err_bit = 3;
  LAUNCH(MT_KERNEL_ENCODE, launch_gemm(bf, &px, 1, EPI_STORE, st));
  LAUNCH(MT_KERNEL_ENCODE, launch_fill_zero(uz, (long long)B * 3 * H, st));
  float *c32 = bf ? nullptr : (float *)ctx_out;
  bf16 *c16 = bf ? (bf16 *)ctx_out : nullptr;
  const int Te = model->cfg.enc_transitions;
  float *tx = (float *)(W + L.tx);  // intermediate transition states [dir][B][H]
  float *const *eln = model->cfg.enc_layer_norm ? model->ln_enc : nullptr;
  const float eps = model->cfg.ln_eps;
  for (int n = 0; n < S; ++n) {
    const int pos[2] = {n, S - 1 - n};       // forward, backward position of this pass
    const int prv[2] = {n - 1, S - n};       // the position each direction comes from
    // the output of block i (0: the input block, 1..Te: the transition blocks) of direction d:
    // the final one lands where the next position reads the state from; intermediate ones
    // alternate with it through tx, so a block never reads and writes the same buffer
    struct Slot {
      float *p;
      int ld;
    };
    auto block_out = [&](int d, int i) -> Slot {
      if ((Te - i) % 2 != 0) return {tx + (size_t)d * B * H, H};
      if (bf) return {sst + ((size_t)(2 * d + (n & 1)) * B) * H, H};
      return {c32 + (size_t)pos[d] * C + (size_t)d * H, (int)ldc};
    };
    // recurrent products of both directions from the previous states (zero at n = 0)
    if (n > 0) {
      GemmProblem pr[2]{};
      for (int d = 0; d < 2; ++d) {
        const size_t o = (size_t)prv[d] * C + (size_t)d * H;
        pr[d].A = bf ? (const void *)(c16 + o) : (const void *)(c32 + o);
        pr[d].a_rows = B; pr[d].lda = (int)ldc; pr[d].a_bf16 = bf;
        const Packed &U = d == 0 ? model->wenc_f : model->wenc_b;
        pr[d].Bp = U.p; pr[d].ldb = U.ldb; pr[d].wblk = U.blk;
        pr[d].out = d == 0 ? uf : ub; pr[d].ldc = 3 * H; pr[d].M = B; pr[d].N = 3 * H; pr[d].K = H;
      }
      LAUNCH(MT_KERNEL_ENCODE, launch_gemm(bf, pr, 2, EPI_STORE, st));
    }
    // one launch runs both directions' cells (the second at element offsets from the first)
    struct CellArgs {
      const float *a, *u, *h;
      float *out;
      bf16 *o16;
      const float *keep;
    };
    auto pair_of = [](const CellArgs &f, const CellArgs &b, long long dln) {
      CellPair pr{};
      pr.da = b.a - f.a; pr.du = b.u - f.u; pr.dh = f.h ? b.h - f.h : 0; pr.dout = b.out - f.out;
      pr.d16 = f.o16 ? b.o16 - f.o16 : 0; pr.dkeep = b.keep - f.keep; pr.dln = dln;
      return pr;
    };
    {
      CellArgs ca[2];
      int ldh = 0;
      for (int d = 0; d < 2; ++d) {
        const size_t oc = (size_t)pos[d] * C + (size_t)d * H, op = (size_t)prv[d] * C + (size_t)d * H;
        const float *hsrc;
        if (bf) {
          hsrc = n > 0 ? sst + ((size_t)(2 * d + ((n - 1) & 1)) * B) * H : nullptr;
          ldh = H;
        } else {
          hsrc = n > 0 ? c32 + op : nullptr;
          ldh = (int)ldc;
        }
        ca[d] = {xe + (size_t)pos[d] * 6 * H + (size_t)d * 3 * H, n > 0 ? (d == 0 ? uf : ub) : uz, hsrc,
                 block_out(d, 0).p, bf && Te == 0 ? c16 + oc : nullptr, mask + pos[d]};
      }
      const CellPair pr = pair_of(ca[0], ca[1], 3 * H);
      LAUNCH(MT_KERNEL_ENCODE,
             launch_gru_cell_ex(B, H, ca[0].a, S * 6 * H, nullptr, B, ca[0].u, 3 * H, ca[0].h, ldh, nullptr, B,
                                model->err, eln ? eln[0] : nullptr, eln ? eln[1] : nullptr, eln ? eln[2] : nullptr,
                                eln ? eln[3] : nullptr, eps, ca[0].out, block_out(0, 0).ld, ca[0].o16, (int)ldc,
                                nullptr, ca[0].keep, S, st, &pr));
    }
    // transition blocks: recurrent products of both directions, then both directions' cells
    // with the bias as the whole input path (lda = 0); a padded position keeps its state
    for (int j = 0; j < Te; ++j) {
      GemmProblem pt[2]{};
      for (int d = 0; d < 2; ++d) {
        const Slot x = block_out(d, j);
        pt[d].A = x.p; pt[d].a_rows = B; pt[d].lda = x.ld; pt[d].a_bf16 = 0;
        const Packed &U = d == 0 ? model->wenc_tf[j] : model->wenc_tb[j];
        pt[d].Bp = U.p; pt[d].ldb = U.ldb; pt[d].wblk = U.blk;
        pt[d].out = d == 0 ? uf : ub; pt[d].ldc = 3 * H; pt[d].M = B; pt[d].N = 3 * H; pt[d].K = H;
      }
      LAUNCH(MT_KERNEL_ENCODE, launch_gemm(bf, pt, 2, EPI_STORE, st));
      CellArgs ca[2];
      for (int d = 0; d < 2; ++d) {
        const size_t oc = (size_t)pos[d] * C + (size_t)d * H;
        ca[d] = {model->bias_tenc + (size_t)(2 * j + d) * 3 * H, d == 0 ? uf : ub, block_out(d, j).p,
                 block_out(d, j + 1).p, bf && j + 1 == Te ? c16 + oc : nullptr, mask + pos[d]};
      }
      const CellPair pr = pair_of(ca[0], ca[1], (long long)Te * 3 * H);
      const size_t to = (size_t)j * 3 * H;  // forward direction's block j
      LAUNCH(MT_KERNEL_ENCODE,
             launch_gru_cell_ex(B, H, ca[0].a, 0, nullptr, B, ca[0].u, 3 * H, ca[0].h, block_out(0, j).ld, nullptr,
                                B, model->err, nullptr, nullptr, eln ? eln[4] + to : nullptr,
                                eln ? eln[5] + to : nullptr, eps, ca[0].out, block_out(0, j + 1).ld, ca[0].o16,
                                (int)ldc, nullptr, ca[0].keep, S, st, &pr));
    }
  }
  return MT_OK;
}

// The precompute's launches on a workspace of at least precompute_ws_bytes (validated by the
// caller).  timed = false launches without the profiling events (the no-alloc entry point).
static mt_status precompute_impl(mt_model *model, int B, int S, const void *ctx, const float *mask, void *pctx_out,
                                 float *s0_out, void *ws, hipStream_t st, bool timed) {
  model->shadow_of = nullptr;
  const mt_config &c = model->cfg;
  const int H = c.H, A = c.A, C = model->C;
  float *cbar = (float *)ws;
  int32_t *vrows = (int32_t *)((char *)ws + rup256((size_t)B * C * 4));
  int *nvalid = (int *)((char *)vrows + rup256((size_t)B * S * 4));
  // keys only at valid positions (the others are never read): the product gathers the valid
  // context rows, counted on the device, and stores each key row at its own position
  LAUNCH_IF(MT_KERNEL_PRECOMPUTE, timed, launch_valid_rows(B * S, mask, vrows, nvalid, st));
  GemmProblem p{};
  p.A = ctx; p.a_idx = vrows; p.a_rows = B * S; p.lda = C; p.a_bf16 = model->bf16;
  p.Bp = model->wp.p; p.ldb = model->wp.ldb; p.wblk = model->wp.blk; p.bias = model->ba;
  p.out = pctx_out; p.ldc = A; p.out_bf16 = model->bf16;
  p.M = B * S; p.N = A; p.K = C; p.err = nullptr; p.err_bit = 0; p.m_dev = nvalid;
  LAUNCH_IF(MT_KERNEL_PRECOMPUTE, timed, launch_gemm(model->bf16, &p, 1, EPI_SCATTER, st));
  LAUNCH_IF(MT_KERNEL_PRECOMPUTE, timed, launch_masked_mean(B, S, C, ctx, model->bf16, mask, cbar, st));
  GemmProblem q{};
  q.A = cbar; q.a_rows = B; q.lda = C; q.a_bf16 = 0;
  q.Bp = model->ws0.p; q.ldb = model->ws0.ldb; q.wblk = model->ws0.blk; q.bias = model->bi;
  q.out = s0_out; q.ldc = H; q.out_bf16 = 0;
  q.M = B; q.N = H; q.K = C;
  LAUNCH_IF(MT_KERNEL_PRECOMPUTE, timed, launch_gemm(model->bf16, &q, 1, EPI_TANH, st));
  // the batch's sentence order for the steps' attention (into model memory)
  if (B <= attention_order_max_sentences()) {
    LAUNCH_IF(MT_KERNEL_PRECOMPUTE, timed, launch_attention_order(B, S, mask, model->srank[0], st));
    model->srank_B[0] = B;
  } else {
    model->srank_B[0] = -1;
  }
  return MT_OK;
}

static mt_status precompute_args(mt_model *model, int B, int S, const void *ctx, const float *mask,
                                 const void *pctx_out, const float *s0_out) {
  if (!valid_model(model)) return fail(MT_ERR_ARG, "invalid model handle");
  if (B < 1 || S < 1 || S > 1024) return fail(MT_ERR_SHAPE, "B=%d S=%d: need B >= 1, 1 <= S <= 1024", B, S);
  if ((long long)B * S > (1 << 24)) return fail(MT_ERR_SHAPE, "B*S=%lld exceeds 2^24", (long long)B * S);
  CHECK(check_dev_ptr(ctx, "ctx"));
  CHECK(check_dev_ptr(mask, "mask", 4));
  CHECK(check_dev_ptr(pctx_out, "pctx_out"));
  CHECK(check_dev_ptr(s0_out, "s0_out"));
  return MT_OK;
}

mt_status mt_precompute_ctx(mt_model *model, int B, int S, const void *ctx, const float *mask,
                            void *pctx_out, float *s0_out, void *ws, size_t ws_bytes, void *stream) {
  g_err[0] = 0;
  CHECK(precompute_args(model, B, S, ctx, mask, pctx_out, s0_out));
  CHECK(check_dev_ptr(ws, "ws", 256));
  const size_t need = precompute_ws_bytes(model, B, S);
  if (ws_bytes < need) return fail(MT_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, need);
  return precompute_impl(model, B, S, ctx, mask, pctx_out, s0_out, ws, (hipStream_t)stream, true);
}

mt_status mt_precompute_ctx_noalloc(mt_model *model, int B, int S, const void *ctx, const float *mask,
                                    void *pctx_out, float *s0_out, void *stream) {
  g_err[0] = 0;
  CHECK(precompute_args(model, B, S, ctx, mask, pctx_out, s0_out));
  const size_t need = precompute_ws_bytes(model, B, S);
  if (need > kNoAllocScratchBytes)
    return fail(MT_ERR_WORKSPACE, "B=%d S=%d needs %zu bytes of scratch, more than the %zu of the no-alloc entry point",
                B, S, need, kNoAllocScratchBytes);
  int dev = -1;
  HIP_TRY(hipGetDevice(&dev));
  if (dev != model->device)
    return fail(MT_ERR_STATE, "current device %d is not the model's device %d", dev, model->device);
  void *sp = nullptr;
  CHECK(scratch_for_device(dev, &sp));
  // every scratch byte the kernels read they first write (valid-row list and count, masked
  // means), so nothing is cleared: what the previous call left is never read
  return precompute_impl(model, B, S, ctx, mask, pctx_out, s0_out, sp, (hipStream_t)stream, false);
}

// The step, with an optional second source (S2 > 0: dual-source models)
// ens_w != 0: a fused-ensemble member: logp_out receives ens_w * logits, added to what it holds
// when ens_acc, and is not turned into log-probabilities.  Only the last member (ens_last: the
// ensemble's size) collects beam candidates, on the combined values it stores; the others
// skip the threshold pass and write only their log-sum-exp partials.  With logp_out NULL the
// member stops after the threshold sample: the joint pass of mt_ensemble_topk does the rest.
static mt_status decoder_step_impl(mt_model *model, int B, int K, int S, const int32_t *prev_tok,
                                   const int32_t *src_row, int n_state_rows, const float *state_in,
                                   const void *ctx, const void *pctx, const float *mask, int S2, const void *ctx2,
                                   const void *pctx2, const float *mask2, float *state_out, float *logp_out,
                                   float *attn_out, const mt_taps *taps, void *ws, size_t ws_bytes, void *stream,
                                   float ens_w = 0.f, int ens_acc = 0, int ens_last = 0) {
  const mt_config &c = model->cfg;
  if (B < 1 || K < 1 || K > c.k_max || K > c.V || S < 1 || S > 1024)
    return fail(MT_ERR_SHAPE, "B=%d K=%d S=%d: need B >= 1, 1 <= K <= k_max=%d, 1 <= S <= 1024", B, K, S, c.k_max);
  if ((long long)B * K > (1 << 20)) return fail(MT_ERR_SHAPE, "B*K exceeds 2^20");
  if ((long long)B * S > (1 << 24)) return fail(MT_ERR_SHAPE, "B*S exceeds 2^24");
  if (n_state_rows < 1) return fail(MT_ERR_SHAPE, "n_state_rows=%d must be >= 1", n_state_rows);
  CHECK(check_dev_ptr(prev_tok, "prev_tok", 4));
  CHECK(check_dev_ptr(src_row, "src_row", 4));
  CHECK(check_dev_ptr(state_in, "state_in"));
  CHECK(check_dev_ptr(ctx, "ctx"));
  CHECK(check_dev_ptr(pctx, "pctx"));
  CHECK(check_dev_ptr(mask, "mask", 4));
  CHECK(check_dev_ptr(state_out, "state_out"));
  CHECK(check_dev_ptr(ws, "ws", 256));
  if (logp_out) CHECK(check_dev_ptr(logp_out, "logp_out", 4));
  if (attn_out) CHECK(check_dev_ptr(attn_out, "attn_out", 4));
  if (taps) {
    if (taps->s1) CHECK(check_dev_ptr(taps->s1, "taps->s1", 4));
    if (taps->c) CHECK(check_dev_ptr(taps->c, "taps->c", 4));
    if (taps->t) CHECK(check_dev_ptr(taps->t, "taps->t", 4));
  }
  const int M = B * K, E = c.E, H = c.H, A = c.A, V = c.V, C = model->C;
  const int nsrc = S2 > 0 ? 2 : 1;
  const int Cc = nsrc * C, ldg2 = nsrc * A + 3 * H;  // context width, s1-product width
  {
    const char *si = (const char *)state_in, *so = (const char *)state_out;
    if (si < so + (size_t)M * H * 4 && so < si + (size_t)n_state_rows * H * 4)
      return fail(MT_ERR_ARG, "state_out overlaps state_in");
  }
  const WsLayout L = ws_layout(model, B, K);
  if (ws_bytes < L.total) return fail(MT_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, L.total);
  hipStream_t st = (hipStream_t)stream;
  char *W = (char *)ws;
  float *gh = (float *)(W + L.gh), *s1 = (float *)(W + L.s1);
  float *g2 = (float *)(W + L.g2), *cc = (float *)(W + L.c), *g3 = (float *)(W + L.g3);
  float *g4 = (float *)(W + L.g4);
  void *t = W + L.t;
  const int bf = model->bf16;
  const float eps = c.ln_eps;
  float *const *ln = model->ln;
  const bool LNon = c.layer_norm != 0;

  // GRU 1: h U1 (the gathered previous state), then the cell with the token side gathered
  // from the precomputed x [W1 | Wt_y] + [b1 | 0] table
  GemmProblem p1{};
  // bf16 models under mt_set_state_reuse: when state_in is the previous step's state_out on
  // this workspace, the product gathers the bf16 copy of it that step left there (the very
  // values it would round state_in to)
  const bool shadow = bf && model->reuse_state && state_in == model->shadow_of && ws == model->shadow_ws &&
                      n_state_rows == model->shadow_rows;
  model->shadow_of = nullptr;  // valid again only once this step has completed its launches
  p1.A = shadow ? (const void *)(W + L.sth) : (const void *)state_in;
  p1.a_idx = src_row; p1.a_rows = n_state_rows; p1.lda = H; p1.a_bf16 = shadow ? 1 : 0;
  p1.Bp = model->w1h.p; p1.ldb = model->w1h.ldb; p1.wblk = model->w1h.blk; p1.bias = nullptr;
  p1.out = gh; p1.ldc = 3 * H; p1.M = M; p1.N = 3 * H; p1.K = H;
  p1.err = model->err; p1.err_bit = 1;
  LAUNCH(MT_KERNEL_GEMM_GRU1, launch_gemm(bf, &p1, 1, EPI_STORE, st));
  LAUNCH(MT_KERNEL_GRU_CELL,
         launch_gru_cell(M, H, model->embx, 3 * H + E, prev_tok, V, gh, 3 * H, state_in, src_row, n_state_rows,
                         model->err, LNon ? ln[0] : nullptr, ln[1], ln[2], ln[3], eps, s1, H,
                         bf ? (bf16 *)(W + L.s1h) : nullptr, taps ? taps->s1 : nullptr, st));
  // s1 [Wa | U2]: attention query and GRU 2 recurrent product (bf16 models read the bf16 copy
  // of s1, which holds exactly the values the product would round s1 to)
  GemmProblem p2{};
  p2.A = bf ? (const void *)(W + L.s1h) : (const void *)s1; p2.a_rows = M; p2.lda = H; p2.a_bf16 = bf;
  p2.Bp = model->w2.p; p2.ldb = model->w2.ldb; p2.wblk = model->w2.blk;
  p2.out = g2; p2.ldc = ldg2; p2.M = M; p2.N = ldg2; p2.K = H;
  LAUNCH(MT_KERNEL_GEMM_S1, launch_gemm(bf, &p2, 1, EPI_STORE, st));
  // bf16 models need the context only in bf16 (fp32 too when it is tapped); a second source's
  // context goes to the right half of the [M][2C] rows
  float *cc32 = (!bf || (taps && taps->c)) ? cc : nullptr;
  bf16 *ch = bf ? (bf16 *)(W + L.ch) : nullptr;
  // rows are scheduled longest sentence first, by the order the batch's precompute left in the
  // model (any permutation of the B sentences gives the same results: it only schedules)
  const int *srank1 = model->srank_B[0] == B ? model->srank[0] : nullptr;
  const int *srank2 = model->srank_B[1] == B ? model->srank[1] : nullptr;
  LAUNCH(MT_KERNEL_ATTENTION, launch_attention(B, K, S, A, C, pctx, ctx, bf, mask, g2, ldg2, model->va, cc32, Cc,
                                               ch, Cc, attn_out, srank1, st));
  if (S2 > 0)
    LAUNCH(MT_KERNEL_ATTENTION, launch_attention(B, K, S2, A, C, pctx2, ctx2, bf, mask2, g2 + A, ldg2, model->va2,
                                                 cc32 ? cc32 + C : nullptr, Cc, ch ? ch + C : nullptr, Cc, nullptr,
                                                 srank2, st));
  if (taps && taps->c) HIP_TRY(hipMemcpyAsync(taps->c, cc, (size_t)M * Cc * 4, hipMemcpyDeviceToDevice, st));
  // c [W2 | Wt_c] + [b2 | 0]
  GemmProblem p3{};
  p3.A = bf ? (const void *)ch : (const void *)cc; p3.a_rows = M; p3.lda = Cc; p3.a_bf16 = bf;
  p3.Bp = model->w3.p; p3.ldb = model->w3.ldb; p3.wblk = model->w3.blk; p3.bias = model->bias3;
  p3.out = g3; p3.ldc = 3 * H + E; p3.M = M; p3.N = 3 * H + E; p3.K = Cc;
  LAUNCH(MT_KERNEL_GEMM_CTX, launch_gemm(bf, &p3, 1, EPI_STORE, st));
  // GRU 2, then the transition blocks of a deep-transition cell (recurrent product s Ut_j,
  // then the cell with the bias row as its input path), alternating between state_out and a
  // workspace buffer so that the last block writes state_out
  const int T = c.dec_transitions;
  float *sx = (float *)(W + L.sx);
  auto dest = [&](int i) { return ((T - i) % 2 == 0) ? state_out : sx; };  // output of block i (0: GRU 2)
  LAUNCH(MT_KERNEL_GRU_CELL,
         launch_gru_cell(M, H, g3, 3 * H + E, nullptr, M, g2 + nsrc * A, ldg2, s1, nullptr, M, model->err,
                         LNon ? ln[4] : nullptr, ln[5], ln[6], ln[7], eps, dest(0), H,
                         bf ? (bf16 *)(W + L.sth) : nullptr, nullptr, st));
  for (int j = 0; j < T; ++j) {
    GemmProblem pt{};
    pt.A = bf ? (const void *)(W + L.sth) : (const void *)dest(j); pt.a_rows = M; pt.lda = H; pt.a_bf16 = bf;
    pt.Bp = model->wtr[j].p; pt.ldb = model->wtr[j].ldb; pt.wblk = model->wtr[j].blk;
    pt.out = gh; pt.ldc = 3 * H; pt.M = M; pt.N = 3 * H; pt.K = H;
    LAUNCH(MT_KERNEL_GEMM_TRANSITION, launch_gemm(bf, &pt, 1, EPI_STORE, st));
    const size_t o = (size_t)j * 3 * H;
    LAUNCH(MT_KERNEL_GRU_CELL,
           launch_gru_cell(M, H, model->btr + o, 0, nullptr, 1, gh, 3 * H, dest(j), nullptr, M, model->err,
                           nullptr, nullptr, LNon ? model->gtu + o : nullptr, LNon ? model->betu + o : nullptr,
                           eps, dest(j + 1), H, bf ? (bf16 *)(W + L.sth) : nullptr, nullptr, st));
  }
  // readout: s Wt_s, then tanh(LN?(s Wt_s + x Wt_y + c Wt_c + bt))
  GemmProblem p4{};
  p4.A = bf ? (const void *)(W + L.sth) : (const void *)state_out; p4.a_rows = M; p4.lda = H; p4.a_bf16 = bf;
  p4.Bp = model->w4.p; p4.ldb = model->w4.ldb; p4.wblk = model->w4.blk;
  p4.out = g4; p4.ldc = E; p4.M = M; p4.N = E; p4.K = H;
  LAUNCH(MT_KERNEL_GEMM_READOUT, launch_gemm(bf, &p4, 1, EPI_STORE, st));
  LAUNCH(MT_KERNEL_READOUT, launch_readout(M, E, g4, E, model->embx + 3 * H, 3 * H + E, prev_tok, V, g3 + 3 * H,
                                           3 * H + E, model->bt,
                                           LNon ? ln[8] : nullptr, ln[9], eps, t, bf, taps ? taps->t : nullptr, st));
  // vocabulary projection: threshold pass, then the full pass with fused log-sum-exp partials
  // and threshold-filtered beam candidates
  float2 *part = (float2 *)(W + L.part);
  const bool ens = ens_w != 0.f;
  const bool joint = ens && !logp_out;
  const bool want_cand = !ens || ens_last > 0;
  if (want_cand || joint) {
    const int S = vocab_sample_size(V);
    GemmProblem ps{};
    ps.A = t; ps.a_rows = M; ps.lda = E; ps.a_bf16 = bf;
    ps.Bp = model->wsamp.p; ps.ldb = model->wsamp.ldb; ps.wblk = model->wsamp.blk; ps.bias = model->bo_pad;
    ps.out = W + L.sample; ps.ldc = S; ps.M = M; ps.N = S; ps.K = E;
    LAUNCH(MT_KERNEL_VOCAB_THRESHOLD, launch_gemm(bf, &ps, 1, EPI_STORE, st));
    if (!joint)
      LAUNCH(MT_KERNEL_VOCAB_THRESHOLD,
             launch_vocab_threshold(M, V, K, (const float *)(W + L.sample), (float *)(W + L.thr),
                                    (int *)(W + L.scnt), B, st, ens && ens_acc ? logp_out : nullptr,
                                    ens ? ens_w : 1.f));
  }
  if (!joint)
    LAUNCH(MT_KERNEL_VOCAB_GEMM, launch_vocab(bf, t, model->wo_frag, model->bo_pad, M, V, E, L.ntiles,
                                              want_cand ? (const float *)(W + L.thr) : nullptr, part,
                                              (int2 *)(W + L.cbuf), (int *)(W + L.ccnt), kVocabCap, logp_out,
                                              model->logit_bounded, st, ens ? ens_w : 1.f, ens_acc, ens ? 1 : 0));
  // the row log-sum-exp is merged by the beam selection itself; this pass only turns the
  // written logits into log-probabilities
  if (logp_out && !ens)
    LAUNCH(MT_KERNEL_LSE, launch_lse(M, L.ntiles, part, (float *)(W + L.lse), logp_out, V, st));
  model->last_B = B;
  model->last_K = K;
  model->last_ws = ws;
  model->shadow_of = bf ? state_out : nullptr;  // the step's bf16 copy of state_out is in L.sth
  model->shadow_ws = ws;
  model->shadow_rows = M;
  model->last_ens_n = ens ? ens_last : 0;
  model->last_ens_w = ens_w;
  model->last_ens_joint = 0;  // set by mt_ensemble_step
  return MT_OK;
}

mt_status mt_decoder_step(mt_model *model, int B, int K, int S, const int32_t *prev_tok,
                          const int32_t *src_row, int n_state_rows, const float *state_in,
                          const void *ctx, const void *pctx, const float *mask, float *state_out,
                          float *logp_out, float *attn_out, const mt_taps *taps, void *ws,
                          size_t ws_bytes, void *stream) {
  g_err[0] = 0;
  if (!valid_model(model)) return fail(MT_ERR_ARG, "invalid model handle");
  if (model->cfg.dual_source) return fail(MT_ERR_STATE, "dual-source model: use mt_decoder_step_dual");
  return decoder_step_impl(model, B, K, S, prev_tok, src_row, n_state_rows, state_in, ctx, pctx, mask, 0, nullptr,
                           nullptr, nullptr, state_out, logp_out, attn_out, taps, ws, ws_bytes, stream);
}

mt_status mt_decoder_step_dual(mt_model *model, int B, int K, int S, const int32_t *prev_tok,
                               const int32_t *src_row, int n_state_rows, const float *state_in,
                               const void *ctx, const void *pctx, const float *mask, int S2, const void *ctx2,
                               const void *pctx2, const float *mask2, float *state_out, float *logp_out,
                               float *attn_out, const mt_taps *taps, void *ws, size_t ws_bytes, void *stream) {
  g_err[0] = 0;
  if (!valid_model(model)) return fail(MT_ERR_ARG, "invalid model handle");
  if (!model->cfg.dual_source) return fail(MT_ERR_STATE, "not a dual-source model (dual_source = 0)");
  if (S2 < 1 || S2 > 1024) return fail(MT_ERR_SHAPE, "S2=%d: need 1 <= S2 <= 1024", S2);
  if ((long long)B * S2 > (1 << 24)) return fail(MT_ERR_SHAPE, "B*S2 exceeds 2^24");
  CHECK(check_dev_ptr(ctx2, "ctx2"));
  CHECK(check_dev_ptr(pctx2, "pctx2"));
  CHECK(check_dev_ptr(mask2, "mask2", 4));
  return decoder_step_impl(model, B, K, S, prev_tok, src_row, n_state_rows, state_in, ctx, pctx, mask, S2, ctx2,
                           pctx2, mask2, state_out, logp_out, attn_out, taps, ws, ws_bytes, stream);
}

// The joint vocabulary pass of a fused ensemble and its selection: the combined threshold, one
// vocabulary kernel for all members (their readout activations and threshold samples are in
// their workspaces), the row constant, then the selection from the combined candidates.
// Candidates, threshold and the selection's scratch live in ws[0].  Arguments checked.
static mt_status ensemble_topk_joint(int n, mt_model *const *models, const float *weights, void *const *ws, int B,
                                     int K, const float *prev_score, float *score_out, int32_t *tok_out,
                                     int32_t *bp_out, int32_t *row_out, float *row_const_out, hipStream_t st) {
  mt_model *model = models[0];  // profiling slot
  const mt_config &c = model->cfg;
  const int M = B * K, V = c.V, E = c.E, bf = model->bf16;
  if (n < 2 || n > kJointMax || vocab_joint_rows(bf, E, n) == 0)
    return fail(MT_ERR_SHAPE, "the joint vocabulary pass does not support %d members at E=%d", n, E);
  const int nj = vocab_joint_chunks(bf, M, V, E, n, model->num_cu);
  const WsLayout L0 = ws_layout(model, B, K);
  char *W0 = (char *)ws[0];
  VocabJointSample smp{};
  smp.n = n;
  smp.ld = vocab_sample_size(V);
  VocabJoint vj{};
  vj.n = n; vj.bf16_mma = bf; vj.M = M; vj.V = V; vj.E = E; vj.n_chunks = nj; vj.cap = kVocabCap;
  vj.fixed_ref = 1;
  EnsembleConst ec{};
  ec.n = n;
  RowSelect rs{};
  rs.nens = n;
  for (int i = 0; i < n; ++i) {
    mt_model *mi = models[i];
    const WsLayout Li = ws_layout(mi, B, K);
    if (nj > Li.ntiles) return fail(MT_ERR_STATE, "member %d: workspace holds %d chunks < %d", i, Li.ntiles, nj);
    char *Wi = (char *)ws[i];
    smp.sample[i] = (const float *)(Wi + Li.sample);
    smp.w[i] = weights[i];
    vj.t[i] = Wi + Li.t;
    vj.wp[i] = mi->wo_frag;
    vj.bias[i] = mi->bo_pad;
    vj.w[i] = weights[i];
    vj.part[i] = (float2 *)(Wi + Li.part);
    vj.fixed_ref &= mi->logit_bounded ? 1 : 0;
    ec.part[i] = vj.part[i];
    ec.ntiles[i] = nj;
    ec.w[i] = weights[i];
    rs.evv[i].t = vj.t[i]; rs.evv[i].wp = mi->wo_frag; rs.evv[i].bias = mi->bo_pad;
    rs.evv[i].V = V; rs.evv[i].E = E; rs.evv[i].KS = E / (bf ? 16 : 8);
    rs.ew[i] = weights[i];
  }
  float *thr = (float *)(W0 + L0.thr);
  int *scnt = (int *)(W0 + L0.scnt);
  LAUNCH(MT_KERNEL_VOCAB_THRESHOLD, launch_vocab_joint_threshold(M, V, K, smp, thr, scnt, B, st));
  vj.thr = thr;
  vj.cbuf = (int2 *)(W0 + L0.cbuf);
  vj.ccnt = (int *)(W0 + L0.ccnt);
  LAUNCH(MT_KERNEL_VOCAB_GEMM, launch_vocab_joint(vj, st));
  float *prev_adj = (float *)(W0 + L0.lse);  // prev_score - C, in the row log-sum-exp slot
  ec.prev = prev_score;
  ec.prev_adj = prev_adj;
  ec.row_const = row_const_out;
  LAUNCH(MT_KERNEL_ENSEMBLE, launch_ensemble_const(ec, M, st));
  rs.B = B; rs.K = K; rs.V = V;
  rs.nl = nj * vocab_lists(); rs.cap = kVocabCap;
  rs.cnt = vj.ccnt;
  rs.cbuf = vj.cbuf;
  rs.prev_score = prev_adj;
  rs.bf16_mma = bf;
  rs.row_cand = (int2 *)(W0 + L0.rowc);
  rs.scnt = scnt;
  rs.score_out = score_out; rs.tok_out = tok_out; rs.bp_out = bp_out; rs.row_out = row_out;
  rs.nrecompute = model->nrecompute;
  LAUNCH(MT_KERNEL_TOPK, launch_row_select(rs, st));
  return MT_OK;
}

mt_status mt_set_state_reuse(mt_model *model, int on) {
  g_err[0] = 0;
  if (!valid_model(model)) return fail(MT_ERR_ARG, "invalid model handle");
  model->reuse_state = on ? 1 : 0;
  return MT_OK;
}

int mt_ensemble_joint_ok(int n, mt_model *const *models) {
  if (n < 2 || n > kJointMax || !models) return 0;
  for (int i = 0; i < n; ++i) {
    if (!valid_model(models[i]) || models[i]->cfg.dual_source) return 0;
    if (models[i]->cfg.V != models[0]->cfg.V || models[i]->cfg.E != models[0]->cfg.E ||
        models[i]->bf16 != models[0]->bf16)
      return 0;
  }
  return vocab_joint_rows(models[0]->bf16, models[0]->cfg.E, n) > 0 ? 1 : 0;
}

mt_status mt_ensemble_step(mt_model *model, int member, int n_members, float weight, int B, int K, int S,
                           const int32_t *prev_tok,
                           const int32_t *src_row, int n_state_rows, const float *state_in, const void *ctx,
                           const void *pctx, const float *mask, float *state_out, float *comb_logits, void *ws,
                           size_t ws_bytes, void *stream) {
  g_err[0] = 0;
  if (!valid_model(model)) return fail(MT_ERR_ARG, "invalid model handle");
  if (model->cfg.dual_source) return fail(MT_ERR_STATE, "dual-source model: not supported in a fused ensemble");
  if (n_members < 1 || n_members > kMaxEnsemble)
    return fail(MT_ERR_ARG, "n_members=%d: need 1..%d", n_members, kMaxEnsemble);
  if (member < 0 || member >= n_members) return fail(MT_ERR_ARG, "member=%d: need 0..%d", member, n_members - 1);
  if (!(weight != 0.f && std::isfinite(weight))) return fail(MT_ERR_ARG, "weight must be finite and nonzero");
  if (comb_logits) {
    CHECK(check_dev_ptr(comb_logits, "comb_logits", 4));
  } else if (vocab_joint_rows(model->bf16, model->cfg.E, n_members) == 0) {
    return fail(MT_ERR_SHAPE, "the joint vocabulary pass does not support %d members at E=%d (%s): pass comb_logits",
                n_members, model->cfg.E, model->bf16 ? "bf16" : "fp32");
  }
  CHECK(decoder_step_impl(model, B, K, S, prev_tok, src_row, n_state_rows, state_in, ctx, pctx, mask, 0, nullptr,
                          nullptr, nullptr, state_out, comb_logits, nullptr, nullptr, ws, ws_bytes, stream, weight,
                          member > 0 ? 1 : 0, member == n_members - 1 ? n_members : 0));
  model->last_ens_joint = comb_logits ? 0 : n_members;
  return MT_OK;
}

mt_status mt_ensemble_topk(int n, mt_model *const *models, const float *weights, void *const *ws,
                           const size_t *ws_bytes, int B, int K, const float *prev_score, const float *comb_logits,
                           float *score_out, int32_t *tok_out, int32_t *bp_out, int32_t *row_out, float *row_const_out,
                           void *stream) {
  g_err[0] = 0;
  if (n < 1 || n > kMaxEnsemble) return fail(MT_ERR_SHAPE, "n=%d: need 1..%d members", n, kMaxEnsemble);
  if (!models || !weights || !ws || !ws_bytes) return fail(MT_ERR_ARG, "models, weights, ws or ws_bytes is NULL");
  mt_model *lead = models[0];
  if (!valid_model(lead)) return fail(MT_ERR_ARG, "invalid model handle (member 0)");
  const mt_config &c = lead->cfg;
  if (B < 1 || K < 1 || K > c.k_max || K > c.V) return fail(MT_ERR_SHAPE, "B=%d K=%d: need B >= 1, 1 <= K <= k_max", B, K);
  if ((long long)B * K > (1 << 20)) return fail(MT_ERR_SHAPE, "B*K exceeds 2^20");
  CHECK(check_dev_ptr(prev_score, "prev_score", 4));
  const bool joint = comb_logits == nullptr;
  if (!joint) CHECK(check_dev_ptr(comb_logits, "comb_logits", 4));
  CHECK(check_dev_ptr(score_out, "score_out", 4));
  CHECK(check_dev_ptr(tok_out, "tok_out", 4));
  CHECK(check_dev_ptr(bp_out, "bp_out", 4));
  if (row_out) CHECK(check_dev_ptr(row_out, "row_out", 4));
  if (row_const_out) CHECK(check_dev_ptr(row_const_out, "row_const_out", 4));
  EnsembleConst ec{};
  ec.n = n;
  for (int i = 0; i < n; ++i) {
    mt_model *mi = models[i];
    if (!valid_model(mi)) return fail(MT_ERR_ARG, "invalid model handle (member %d)", i);
    if (mi->cfg.V != c.V || mi->cfg.k_max < K) return fail(MT_ERR_SHAPE, "member %d: V or k_max differs", i);
    if (!std::isfinite(weights[i]) || weights[i] == 0.f) return fail(MT_ERR_ARG, "weights[%d] must be finite and nonzero", i);
    CHECK(check_dev_ptr(ws[i], "ws[i]", 256));
    const WsLayout Li = ws_layout(mi, B, K);
    if (ws_bytes[i] < Li.total) return fail(MT_ERR_WORKSPACE, "ws[%d]: %zu bytes < %zu needed", i, ws_bytes[i], Li.total);
    if (mi->last_B != B || mi->last_K != K || mi->last_ws != ws[i] || mi->last_ens_w != weights[i])
      return fail(MT_ERR_STATE, "member %d: no preceding mt_ensemble_step with this B, K, weight and workspace", i);
    if (joint) {
      if (mi->last_ens_joint != n)
        return fail(MT_ERR_STATE, "member %d: its mt_ensemble_step was not a joint-pass step of %d members", i, n);
      if (mi->cfg.E != c.E || mi->bf16 != lead->bf16)
        return fail(MT_ERR_SHAPE, "member %d: E or gemm dtype differs (the joint pass needs them equal)", i);
    } else if (mi->last_ens_joint != 0 || (mi->last_ens_n != 0) != (i == n - 1) ||
               (i == n - 1 && mi->last_ens_n != n)) {
      return fail(MT_ERR_STATE, "member %d: its mt_ensemble_step was not called as member %d of %d", i, i, n);
    }
    ec.part[i] = (const float2 *)((const char *)ws[i] + Li.part);
    ec.ntiles[i] = Li.ntiles;
    ec.w[i] = weights[i];
  }
  if (joint) return ensemble_topk_joint(n, models, weights, ws, B, K, prev_score, score_out, tok_out, bp_out, row_out,
                                         row_const_out, (hipStream_t)stream);
  // the candidates are the last member's (collected on the combined values), and so is the
  // selection's scratch
  mt_model *model = models[n - 1];  // profiling slot
  hipStream_t st = (hipStream_t)stream;
  const WsLayout L = ws_layout(model, B, K);
  char *W = (char *)ws[n - 1];
  const int M = B * K, V = c.V;
  float *prev_adj = (float *)(W + L.lse);  // prev_score - C, in the row log-sum-exp slot
  ec.prev = prev_score;
  ec.prev_adj = prev_adj;
  ec.row_const = row_const_out;
  LAUNCH(MT_KERNEL_ENSEMBLE, launch_ensemble_const(ec, M, st));
  RowSelect rs{};
  rs.B = B; rs.K = K; rs.V = V;
  rs.nl = L.ntiles * vocab_lists(); rs.cap = kVocabCap;
  rs.cnt = (const int *)(W + L.ccnt);
  rs.cbuf = (const int2 *)(W + L.cbuf);
  rs.prev_score = prev_adj;
  rs.comb = comb_logits;
  rs.bf16_mma = model->bf16;
  rs.row_cand = (int2 *)(W + L.rowc);
  rs.scnt = (int *)(W + L.scnt);
  rs.score_out = score_out; rs.tok_out = tok_out; rs.bp_out = bp_out; rs.row_out = row_out;
  rs.nrecompute = model->nrecompute;
  LAUNCH(MT_KERNEL_TOPK, launch_row_select(rs, st));
  return MT_OK;
}

mt_status mt_precompute_keys2(mt_model *model, int B, int S2, const void *ctx2, const float *mask2,
                              void *pctx2_out, void *ws, size_t ws_bytes, void *stream) {
  g_err[0] = 0;
  if (!valid_model(model)) return fail(MT_ERR_ARG, "invalid model handle");
  model->shadow_of = nullptr;
  if (!model->cfg.dual_source) return fail(MT_ERR_STATE, "not a dual-source model (dual_source = 0)");
  if (B < 1 || S2 < 1 || S2 > 1024) return fail(MT_ERR_SHAPE, "B=%d S2=%d: need B >= 1, 1 <= S2 <= 1024", B, S2);
  if ((long long)B * S2 > (1 << 24)) return fail(MT_ERR_SHAPE, "B*S2 exceeds 2^24");
  CHECK(check_dev_ptr(ctx2, "ctx2"));
  CHECK(check_dev_ptr(mask2, "mask2", 4));
  CHECK(check_dev_ptr(pctx2_out, "pctx2_out"));
  CHECK(check_dev_ptr(ws, "ws", 256));
  const size_t need = precompute_ws_bytes(model, B, S2);
  if (ws_bytes < need) return fail(MT_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, need);
  hipStream_t st = (hipStream_t)stream;
  const int A = model->cfg.A, C = model->C;
  int32_t *vrows = (int32_t *)((char *)ws + rup256((size_t)B * C * 4));
  int *nvalid = (int *)((char *)vrows + rup256((size_t)B * S2 * 4));
  LAUNCH(MT_KERNEL_PRECOMPUTE, launch_valid_rows(B * S2, mask2, vrows, nvalid, st));
  GemmProblem p{};
  p.A = ctx2; p.a_idx = vrows; p.a_rows = B * S2; p.lda = C; p.a_bf16 = model->bf16;
  p.Bp = model->wp2.p; p.ldb = model->wp2.ldb; p.wblk = model->wp2.blk; p.bias = model->ba2;
  p.out = pctx2_out; p.ldc = A; p.out_bf16 = model->bf16;
  p.M = B * S2; p.N = A; p.K = C; p.m_dev = nvalid;
  LAUNCH(MT_KERNEL_PRECOMPUTE, launch_gemm(model->bf16, &p, 1, EPI_SCATTER, st));
  if (B <= attention_order_max_sentences()) {
    LAUNCH(MT_KERNEL_PRECOMPUTE, launch_attention_order(B, S2, mask2, model->srank[1], st));
    model->srank_B[1] = B;
  } else {
    model->srank_B[1] = -1;
  }
  return MT_OK;
}

mt_status mt_beam_topk(mt_model *model, int B, int K, const float *prev_score, const float *logp,
                       float *score_out, int32_t *tok_out, int32_t *bp_out, int32_t *row_out,
                       void *ws, size_t ws_bytes, void *stream) {
  g_err[0] = 0;
  if (!valid_model(model)) return fail(MT_ERR_ARG, "invalid model handle");
  const mt_config &c = model->cfg;
  if (B < 1 || K < 1 || K > c.k_max || K > c.V) return fail(MT_ERR_SHAPE, "B=%d K=%d: need B >= 1, 1 <= K <= k_max", B, K);
  if ((long long)B * K > (1 << 20)) return fail(MT_ERR_SHAPE, "B*K exceeds 2^20");
  CHECK(check_dev_ptr(prev_score, "prev_score", 4));
  CHECK(check_dev_ptr(score_out, "score_out", 4));
  CHECK(check_dev_ptr(tok_out, "tok_out", 4));
  CHECK(check_dev_ptr(bp_out, "bp_out", 4));
  if (row_out) CHECK(check_dev_ptr(row_out, "row_out", 4));
  if (logp) CHECK(check_dev_ptr(logp, "logp", 4));
  CHECK(check_dev_ptr(ws, "ws", 256));
  const WsLayout L = ws_layout(model, B, K);
  if (ws_bytes < L.total) return fail(MT_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, L.total);
  if (!logp && (model->last_B != B || model->last_K != K || model->last_ws != ws))
    return fail(MT_ERR_STATE, "no preceding mt_decoder_step with this B, K and workspace (pass logp instead)");
  if (!logp && model->last_ens_w != 0.f)
    return fail(MT_ERR_STATE, "the preceding step was a fused-ensemble member's (select with mt_ensemble_topk)");
  hipStream_t st = (hipStream_t)stream;
  char *W = (char *)ws;
  const int M = B * K, V = c.V;
  int2 *rowc = (int2 *)(W + L.rowc);
  RowSelect rs{};
  rs.B = B; rs.K = K; rs.V = V;
  rs.prev_score = prev_score;
  rs.row_cand = rowc;
  rs.scnt = (int *)(W + L.scnt);
  rs.score_out = score_out; rs.tok_out = tok_out; rs.bp_out = bp_out; rs.row_out = row_out;
  rs.nrecompute = model->nrecompute;
  if (!logp) {
    rs.nl = L.ntiles * vocab_lists(); rs.cap = kVocabCap;
    rs.cnt = (const int *)(W + L.ccnt); rs.cbuf = (const int2 *)(W + L.cbuf);
    rs.part = (const float2 *)(W + L.part); rs.ntiles = L.ntiles;
    rs.vv.t = W + L.t; rs.vv.wp = model->wo_frag; rs.vv.bias = model->bo_pad;
    rs.vv.V = V; rs.vv.E = c.E; rs.vv.KS = c.E / (model->bf16 ? 16 : 8);
    rs.bf16_mma = model->bf16;
    LAUNCH(MT_KERNEL_TOPK, launch_row_select(rs, st));
  } else {
    int2 *sc = (int2 *)(W + L.scand);
    LAUNCH(MT_KERNEL_TOPK, launch_topk_scan_logp(M, K, V, L.nchunks, prev_score, logp, sc, rs.scnt, B, st));
    rs.nl = L.nchunks; rs.cap = K; rs.cbuf = sc;
    LAUNCH(MT_KERNEL_TOPK, launch_row_select(rs, st));
  }
  return MT_OK;
}

mt_status mt_ensemble_logp(mt_model *model, int n, const float *const *logp, const float *weights, int M,
                           float *out, void *stream) {
  g_err[0] = 0;
  if (!valid_model(model)) return fail(MT_ERR_ARG, "invalid model handle");
  if (n < 1 || n > kMaxEnsemble) return fail(MT_ERR_SHAPE, "n=%d: need 1..%d members", n, kMaxEnsemble);
  if (M < 1 || M > (1 << 20)) return fail(MT_ERR_SHAPE, "M=%d: need 1 <= M <= 2^20", M);
  if (!logp || !weights) return fail(MT_ERR_ARG, "logp or weights is NULL");
  for (int i = 0; i < n; ++i) {
    char name[32];
    std::snprintf(name, sizeof name, "logp[%d]", i);
    CHECK(check_dev_ptr(logp[i], name));
    if (!std::isfinite(weights[i])) return fail(MT_ERR_ARG, "weights[%d] is not finite", i);
  }
  CHECK(check_dev_ptr(out, "out"));
  hipStream_t st = (hipStream_t)stream;
  LAUNCH(MT_KERNEL_ENSEMBLE, launch_ensemble(n, logp, weights, (long long)M * model->cfg.V, out, model->num_cu, st));
  return MT_OK;
}

mt_status mt_beam_finish(mt_model *model, int B, int K, int step, int32_t eos, float alpha, int final_step,
                         int32_t *tok, int32_t *bp, int32_t *row, float *score, int32_t *beam,
                         int32_t *fin_count, int32_t *hist_tok, int32_t *hist_bp, float *fin_score,
                         float *fin_norm, int32_t *fin_step, int32_t *fin_parent, int32_t *fin_tok, void *stream) {
  g_err[0] = 0;
  if (!valid_model(model)) return fail(MT_ERR_ARG, "invalid model handle");
  const mt_config &c = model->cfg;
  if (B < 1 || K < 1 || K > c.k_max || K > c.V) return fail(MT_ERR_SHAPE, "B=%d K=%d: need B >= 1, 1 <= K <= k_max", B, K);
  if ((long long)B * K > (1 << 20)) return fail(MT_ERR_SHAPE, "B*K exceeds 2^20");
  if (step < 0) return fail(MT_ERR_ARG, "step=%d must be >= 0", step);
  if (eos < 0 || eos >= c.V) return fail(MT_ERR_ARG, "eos=%d outside [0, V)", eos);
  if (!std::isfinite(alpha)) return fail(MT_ERR_ARG, "alpha is not finite");
  struct {
    const void *p;
    const char *n;
  } ptrs[] = {{tok, "tok"}, {bp, "bp"}, {row, "row"}, {score, "score"}, {beam, "beam"}, {fin_count, "fin_count"},
              {hist_tok, "hist_tok"}, {hist_bp, "hist_bp"}, {fin_score, "fin_score"}, {fin_norm, "fin_norm"},
              {fin_step, "fin_step"}, {fin_parent, "fin_parent"}, {fin_tok, "fin_tok"}};
  for (auto &q : ptrs) CHECK(check_dev_ptr(q.p, q.n, 4));
  hipStream_t st = (hipStream_t)stream;
  BeamFinish a{};
  a.K = K; a.step = step; a.eos = eos; a.final = final_step != 0; a.alpha = alpha;
  a.tok = tok; a.bp = bp; a.row = row; a.score = score; a.beam = beam; a.fin_count = fin_count;
  a.hist_tok = hist_tok; a.hist_bp = hist_bp; a.fin_score = fin_score; a.fin_norm = fin_norm;
  a.fin_step = fin_step; a.fin_parent = fin_parent; a.fin_tok = fin_tok;
  LAUNCH(MT_KERNEL_BEAM_FINISH, launch_beam_finish(a, B, st));
  return MT_OK;
}

mt_status mt_beam_nbest(mt_model *model, int B, int K, int steps, const int32_t *hist_tok, const int32_t *hist_bp,
                        const int32_t *fin_count, const float *fin_norm, const int32_t *fin_step,
                        const int32_t *fin_parent, const int32_t *fin_tok, int32_t *order, int32_t *seq, int ld_seq,
                        void *stream) {
  g_err[0] = 0;
  if (!valid_model(model)) return fail(MT_ERR_ARG, "invalid model handle");
  if (B < 1 || K < 1 || K > kKMax) return fail(MT_ERR_SHAPE, "B=%d K=%d: need B >= 1, 1 <= K <= %d", B, K, kKMax);
  if ((long long)B * K > (1 << 20)) return fail(MT_ERR_SHAPE, "B*K exceeds 2^20");
  if (steps < 1) return fail(MT_ERR_SHAPE, "steps=%d must be >= 1", steps);
  if (ld_seq < steps) return fail(MT_ERR_SHAPE, "ld_seq=%d < steps=%d", ld_seq, steps);
  if ((long long)B * K * ld_seq > (1ll << 31) || (long long)steps * B * K > (1ll << 31))
    return fail(MT_ERR_SHAPE, "records or sequences exceed 2^31 entries");
  struct {
    const void *p;
    const char *n;
  } ptrs[] = {{hist_tok, "hist_tok"}, {hist_bp, "hist_bp"}, {fin_count, "fin_count"}, {fin_norm, "fin_norm"},
              {fin_step, "fin_step"}, {fin_parent, "fin_parent"}, {fin_tok, "fin_tok"}, {order, "order"},
              {seq, "seq"}};
  for (auto &q : ptrs) CHECK(check_dev_ptr(q.p, q.n, 4));
  hipStream_t st = (hipStream_t)stream;
  BeamNbest a{};
  a.K = K; a.steps = steps; a.ld_hist = B * K; a.ld_seq = ld_seq;
  a.hist_tok = hist_tok; a.hist_bp = hist_bp; a.fin_count = fin_count; a.fin_norm = fin_norm;
  a.fin_step = fin_step; a.fin_parent = fin_parent; a.fin_tok = fin_tok; a.order = order; a.seq = seq;
  LAUNCH(MT_KERNEL_BEAM_FINISH, launch_beam_nbest(a, B, st));
  return MT_OK;
}

mt_status mt_device_errors(mt_model *model, int32_t *flags) {
  g_err[0] = 0;
  if (!valid_model(model)) return fail(MT_ERR_ARG, "invalid model handle");
  if (!flags) return fail(MT_ERR_ARG, "flags is NULL");
  HIP_TRY(hipDeviceSynchronize());
  HIP_TRY(hipMemcpy(flags, model->err, 4, hipMemcpyDeviceToHost));
  HIP_TRY(hipMemset(model->err, 0, 4));
  return MT_OK;
}

mt_status mt_recomputed_rows(mt_model *model, int64_t *rows) {
  g_err[0] = 0;
  if (!valid_model(model)) return fail(MT_ERR_ARG, "invalid model handle");
  if (!rows) return fail(MT_ERR_ARG, "rows is NULL");
  unsigned long long n = 0;
  HIP_TRY(hipDeviceSynchronize());
  HIP_TRY(hipMemcpy(&n, model->nrecompute, sizeof n, hipMemcpyDeviceToHost));
  HIP_TRY(hipMemset(model->nrecompute, 0, sizeof n));
  *rows = (int64_t)n;
  return MT_OK;
}

mt_status mt_profile_enable(mt_model *model, uint32_t kernel_mask) {
  g_err[0] = 0;
  if (!valid_model(model)) return fail(MT_ERR_ARG, "invalid model handle");
  if (kernel_mask >> MT_KERNEL_COUNT) return fail(MT_ERR_ARG, "kernel_mask 0x%x has bits beyond the kernel ids", kernel_mask);
  model->prof_mask = kernel_mask;
  return MT_OK;
}

mt_status mt_profile_sample(mt_model *model, uint32_t every) {
  g_err[0] = 0;
  if (!valid_model(model)) return fail(MT_ERR_ARG, "invalid model handle");
  if (every < 1) return fail(MT_ERR_ARG, "every=%u must be >= 1", every);
  model->prof_every = every;
  return MT_OK;
}

mt_status mt_profile_reset(mt_model *model) {
  g_err[0] = 0;
  if (!valid_model(model)) return fail(MT_ERR_ARG, "invalid model handle");
  for (int k = 0; k < MT_KERNEL_COUNT; ++k) {
    fold_profile(model, k);
    model->prof[k].ms = 0.0;
    model->prof[k].n = 0;
    model->prof[k].seen = 0;
  }
  return MT_OK;
}

mt_status mt_profile_query(mt_model *model, int kernel, double *total_ms, int64_t *launches) {
  g_err[0] = 0;
  if (!valid_model(model)) return fail(MT_ERR_ARG, "invalid model handle");
  if (kernel < 0 || kernel >= MT_KERNEL_COUNT) return fail(MT_ERR_ARG, "kernel id %d out of range", kernel);
  if (!total_ms || !launches) return fail(MT_ERR_ARG, "output pointer is NULL");
  fold_profile(model, kernel);
  *total_ms = model->prof[kernel].ms;
  *launches = model->prof[kernel].n;
  return MT_OK;
}

}  // extern "C"
