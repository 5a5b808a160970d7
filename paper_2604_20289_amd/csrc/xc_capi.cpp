// Host side of the C ABI declared in include/xcache.h: argument validation,
// device state, and the launch sequence of one pass.
//
// Device state of a handle (all allocated once at xc_init):
//   weights        per tensor kind, blocks concatenated; Linear weights in the
//                  model dtype as [out][in] (K-contiguous MFMA operands), the
//                  Q/K/V projections stacked into one [3C][C] matrix per block;
//                  biases, gains in float32
//   KV cache       K  [B][H][Lcap][D], V^T [B][H][D][Lcap]; generation n owns
//                  rows [(n mod W) L, (n mod W + 1) L): the visible chunks are
//                  always the prefix [0, min(n+1, W) L), and the next
//                  generation's slot is the oldest one (FIFO for free)
//   residuals      r_hat [S][B][L][C] in the model dtype (Eq. 3)
//   fingerprints   [S][B][n_srows + n_cams][C] float32
//   gate state     EMA (NaN = unset), staleness, skip counts [S][B]; per-pass
//                  skip flags and records [B]
//   activations    h, q, o, u in the model dtype, padded to Mpad rows; x1
//                  and two ping-pong streams (float32 models also stage the
//                  QKV projection in float32 before the QK-norm kernel).
//   rotary tables  (rope = 1) per-token packed grid coordinates and the
//                  (cos, sin) tables; the frame section is rebuilt whenever
//                  the generation index changes
//   cross-attention (cond_len > 0) its weights per block, the condition's
//                  keys K_c [B][H][Lcap_c][D] and V_c^T [B][H][D][Lcap_c],
//                  the condition tokens in the model dtype [Mcpad][C].
//
// One denoising pass enqueues, per block: for a gated block the fingerprint
// reduction and the decision kernel (its flag stays on the device), then the
// skip-add (runs iff the flag is set) and the compute kernels (each returns at
// entry iff the flag is set).  Nothing is copied back to the host.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "xc_internal.h"
#include "xcache.h"

using namespace xc;

// Scratch of xc_forward_chunk_noalloc: the gate's partial records and the
// attention's key-split partials of one pass, in a static array that every
// GPU the library runs on holds (one copy per device, at its own address)
// until the process ends.  In host code `scratch` only names the symbol; its
// device address comes from hipGetSymbolAddress (device_scratch below).
constexpr size_t kStaticScratchBytes = (size_t)XC_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {

// Device address of `scratch` on the current device, looked up once per
// device (null on failure).
unsigned char* device_scratch(int device) {
  static std::mutex mu;
  static unsigned char* addr[64] = {};
  if (device < 0 || device >= 64) return nullptr;
  std::lock_guard<std::mutex> lock(mu);
  if (addr[device] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
    addr[device] = reinterpret_cast<unsigned char*>(p);
  }
  return addr[device];
}

}  // namespace

struct ProfRecord {
  int kind;
  hipEvent_t start, stop;
};

// Per-pass workspace of the kernels: the gate's per-workgroup partial records
// and the attention's key-split partials (either the handle's own buffers or
// the static scratch array of xc_forward_chunk_noalloc).
struct PassWs {
  double* records;
  float* attn;
  size_t attn_floats;
  bool prof;   // false: record no kernel timings (xc_profile) in this pass
};

struct xc_handle {
  xc_model_config m;
  xc_gate_config g;
  hipStream_t st = nullptr;
  int device = 0;
  int B = 0, C = 0, H = 0, D = 0, Dm = 0, Dt = 0, A = 0, Dc = 0, S = 0, Wkv = 0, dtype = 0;
  long long L = 0, Mpad = 0, Lcap = 0;
  size_t esz = 4;

  // weights
  void* w_ada = nullptr; float* b_ada = nullptr;
  void* wqkv = nullptr; float* bqkv = nullptr; float* gq = nullptr; float* gk = nullptr;
  void* wo = nullptr; float* bo = nullptr; void* w1 = nullptr; float* b1 = nullptr;
  void* w2 = nullptr; float* b2 = nullptr;
  // rotary embedding
  float2* rope_tab = nullptr; int* rope_pos = nullptr; int* rope_slot_frames = nullptr; int* rope_slot_frame = nullptr;
  RopeArgs rope{};
  int rope_slots = 0, rope_rows = 0, rope_cols = 0;
  // cross-attention
  int Mc = 0, n_cond = 0;
  long long Mcpad = 0, Lcap_c = 0;
  void* wqkv_c = nullptr; float* bqkv_c = nullptr; float* gq_c = nullptr; float* gk_c = nullptr;
  void* wo_c = nullptr; float* bo_c = nullptr; float* ln3_shift = nullptr; float* ln3_scale = nullptr;
  void* kc_c = nullptr; void* vt_c = nullptr; void* cond_act = nullptr; float* cond_kv = nullptr;
  float* ones = nullptr;
  // gate global channel from the MLP-down epilogue (bf16 models whose cameras
  // all have >= 32 tokens): partials, 32-row-block tables, per-pass input sums
  // and per-(t, b) residual sums
  bool fold = false;
  int n_rb = 0;
  float* csum_part = nullptr;
  int* rb_split = nullptr; int* rb_cam = nullptr; int* cam_rb_lo = nullptr; int* cam_rb_hi = nullptr;
  double* csum_in = nullptr; double* csum_rhat = nullptr;
  // caches
  void* kc = nullptr; void* vt = nullptr; void* rhat = nullptr; float* fp = nullptr;
  float* fp_alt = nullptr;  // second fingerprint set of the refresh-on-compute mode
  int* fp_sel = nullptr;     // [S][B] which of fp / fp_alt holds the cached fingerprint
  // gate state
  float* ema = nullptr; int* stale = nullptr; int* skip_counts = nullptr; int* flags = nullptr;
  int* rec_dec = nullptr; float* rec_s = nullptr; float* rec_d = nullptr; float* rec_tau = nullptr;
  // activations and scratch
  float* cond = nullptr; float* mod = nullptr;
  void* hbuf = nullptr; float* qkv = nullptr; void* q = nullptr; void* o = nullptr; void* u = nullptr;
  float* x1 = nullptr; float* xa = nullptr; float* xb = nullptr;
  double* fp_records = nullptr;
  float* attn_ws = nullptr;
  size_t attn_ws_floats = 0;
  // device address of this GPU's static scratch array (xc_forward_chunk_noalloc)
  unsigned char* scratch = nullptr;
  // fingerprint tables
  FpTables tables{};
  int n_srows = 0, n_cams = 0, fp_rows = 0, n_wg = 0;
  std::vector<int> spatial_count;
  // host state
  long long n = 0;
  std::vector<char> visited;
  long long evals_post_warmup = 0, gated_evals = 0, kv_block_evals = 0;
  int last_step = -1;
  bool any_forward = false;
  float action_prev[kMaxAction] = {};
  bool have_action_prev = false;
  // the action of the current generation, fixed by its first pass: every
  // pass of one chunk (denoising steps and the clean pass) conditions on it
  float action_cur[kMaxAction] = {};
  bool have_action_cur = false;
  bool sticky = false;
  // profiling
  bool profiling = false;
  bool prof_suspended = false;  // set while a pass must not create events
  std::vector<ProfRecord> prof;
  std::vector<hipEvent_t> ev_free;
  std::vector<void*> allocs;
};

namespace {

// largest visible key window (W_kv x L) and largest per-kind column-sum
// partial buffer (bytes) whose kernel offsets fit in 32 bits
constexpr long long kMaxWindowKeys = 1ll << 24;
constexpr long long kMaxPartialBytes = (1ll << 31) - 1;

bool gateable(const xc_handle* h, int b) {
  return h->g.enabled && b >= h->g.front_anchors && b < h->B - h->g.back_anchors;
}

// an action that differs from the one this generation's first pass fixed
bool action_changed(const xc_handle* h, const float* a) {
  return h->have_action_cur && std::memcmp(h->action_cur, a, sizeof(float) * (size_t)h->A) != 0;
}

void fix_action(xc_handle* h, const float* a) {
  if (h->have_action_cur) return;
  std::memcpy(h->action_cur, a, sizeof(float) * (size_t)h->A);
  h->have_action_cur = true;
}

long long tokens_of(const xc_model_config* m) {
  long long L = 0;
  for (int i = 0; i < m->n_groups; ++i) {
    const xc_view_group& g = m->groups[i];
    L += (long long)g.views * g.frames * g.height * g.width;
  }
  return L;
}

xc_status validate_model(const xc_model_config* m) {
  if (!m) return XC_ERR_INVALID_ARG;
  if (m->n_blocks < 1 || m->n_blocks > 4096) return XC_ERR_INVALID_ARG;
  if (m->n_heads < 1 || m->head_dim < 1 || m->hidden != m->n_heads * m->head_dim) return XC_ERR_INVALID_ARG;
  if (m->hidden % 4 != 0 || m->hidden > 4096) return XC_ERR_INVALID_ARG;
  if (m->head_dim > 128) return XC_ERR_UNSUPPORTED;
  if (m->mlp_hidden < 1 || m->mlp_hidden > 65536) return XC_ERR_INVALID_ARG;
  if (m->temb_dim < 2 || m->temb_dim % 2 != 0) return XC_ERR_INVALID_ARG;
  if (m->action_dim < 0 || m->action_dim > XC_MAX_ACTION) return XC_ERR_INVALID_ARG;
  if (m->temb_dim + m->action_dim > XC_MAX_COND) return XC_ERR_INVALID_ARG;
  if (m->dtype != XC_F32 && m->dtype != XC_BF16) return XC_ERR_INVALID_ARG;
  if (m->n_steps < 1 || m->n_steps > 64) return XC_ERR_INVALID_ARG;
  if (m->kv_window < 1 || m->kv_window > 64) return XC_ERR_INVALID_ARG;
  if (m->n_groups < 1 || m->n_groups > XC_MAX_GROUPS) return XC_ERR_INVALID_ARG;
  for (int i = 0; i < m->n_groups; ++i) {
    const xc_view_group& g = m->groups[i];
    if (g.views < 1 || g.frames < 1 || g.height < 1 || g.width < 1) return XC_ERR_INVALID_ARG;
    if ((long long)g.views * g.frames * g.height * g.width > (1ll << 24)) return XC_ERR_INVALID_ARG;
  }
  const long long L = tokens_of(m);
  if (L < 1 || L > (1ll << 24)) return XC_ERR_INVALID_ARG;
  if ((long long)m->kv_window * L > (1ll << 28)) return XC_ERR_INVALID_ARG;
  // shapes whose 32-bit kernel offsets would wrap: the attention kernel's
  // per-thread V^T staging offset spans up to 63 rows of Lcap keys (bf16),
  // the MLP-down epilogue's column-sum partials ceil(L/32) x 2 x C floats
  if ((long long)m->kv_window * L > kMaxWindowKeys) return XC_ERR_UNSUPPORTED;
  if ((L + 31) / 32 * 2 * (long long)m->hidden * 4 > kMaxPartialBytes) return XC_ERR_UNSUPPORTED;
  if (m->dtype == XC_BF16) {
    if (m->head_dim != 64 && m->head_dim != 128) return XC_ERR_UNSUPPORTED;
    if (m->hidden % 128 != 0 || m->mlp_hidden % 128 != 0) return XC_ERR_UNSUPPORTED;
  }
  if (m->rope != 0 && m->rope != 1) return XC_ERR_INVALID_ARG;
  if (m->rope) {
    if (m->head_dim % 2 != 0) return XC_ERR_INVALID_ARG;
    if (!std::isfinite(m->rope_theta) || !(m->rope_theta > 1.f)) return XC_ERR_INVALID_ARG;
    int slots = 0;
    for (int i = 0; i < m->n_groups; ++i) {
      const xc_view_group& g = m->groups[i];
      if (g.height >= 1024 || g.width >= 1024) return XC_ERR_INVALID_ARG;
      slots += g.frames;
      if (slots >= 1024) return XC_ERR_INVALID_ARG;
    }
  }
  if (m->cond_len < 0 || m->cond_len > 4096) return XC_ERR_INVALID_ARG;
  return XC_OK;
}

xc_status validate_gate(const xc_gate_config* g, const xc_model_config* m) {
  if (!g) return XC_ERR_INVALID_ARG;
  if (g->enabled != 0 && g->enabled != 1) return XC_ERR_INVALID_ARG;
  if (g->fp_budget < 1) return XC_ERR_INVALID_ARG;
  if (g->warmup < 1) return XC_ERR_INVALID_ARG;
  if (g->front_anchors < 0 || g->back_anchors < 0) return XC_ERR_INVALID_ARG;
  if (g->adaptive != 0 && g->adaptive != 1) return XC_ERR_INVALID_ARG;
  if (std::isnan(g->tau_floor) || std::isnan(g->margin) || std::isnan(g->tau_cos_fixed) || std::isnan(g->tau_dev) ||
      std::isnan(g->tau_strict0))
    return XC_ERR_INVALID_ARG;
  if (!(g->alpha >= 0.f && g->alpha <= 1.f)) return XC_ERR_INVALID_ARG;
  if (!(g->eps >= 0.f) || std::isinf(g->eps)) return XC_ERR_INVALID_ARG;
  if (g->max_stale < 0) return XC_ERR_INVALID_ARG;
  if (g->step0_mode < XC_STEP0_OFF || g->step0_mode > XC_STEP0_STRICT) return XC_ERR_INVALID_ARG;
  if (g->fp_mode != XC_FP_GRID3D && g->fp_mode != XC_FP_LINSPACE1D) return XC_ERR_INVALID_ARG;
  if (g->fp_refresh != XC_FP_REFRESH_EVERY && g->fp_refresh != XC_FP_REFRESH_ON_COMPUTE) return XC_ERR_INVALID_ARG;
  if (g->kv_protect == 0) return XC_ERR_UNSUPPORTED;
  if (g->kv_protect != 1) return XC_ERR_INVALID_ARG;
  (void)m;
  return XC_OK;
}

// k uniformly spaced indices on [0, dim-1], floored.
void axis_indices(int dim, int k, std::vector<int>& out) {
  out.clear();
  if (k <= 1) {
    out.push_back(0);
    return;
  }
  for (int i = 0; i < k; ++i) out.push_back((int)(((long long)i * (dim - 1)) / (k - 1)));
}

// Sampled token rows of one camera (local indices), Section 2.3.1.
void camera_rows(const xc_view_group& g, int budget, int mode, std::vector<int>& local) {
  const long long T = (long long)g.frames * g.height * g.width;
  local.clear();
  if (T <= budget) {
    for (int i = 0; i < T; ++i) local.push_back(i);
    return;
  }
  std::vector<int> idx;
  if (mode == XC_FP_LINSPACE1D) {
    axis_indices((int)T, (int)std::min<long long>(budget, T), idx);
    local = idx;
    return;
  }
  const double s = std::pow((double)budget / (double)T, 1.0 / 3.0);
  int k[3];
  const int dims[3] = {g.frames, g.height, g.width};
  for (int a = 0; a < 3; ++a) {
    int v = (int)std::floor((double)dims[a] * s + 0.5);
    k[a] = std::min(std::max(v, 1), dims[a]);
  }
  std::vector<int> fi, hi, wi;
  axis_indices(g.frames, k[0], fi);
  axis_indices(g.height, k[1], hi);
  axis_indices(g.width, k[2], wi);
  for (int f : fi)
    for (int y : hi)
      for (int x : wi) local.push_back(f * g.height * g.width + y * g.width + x);
}

void all_rows(const xc_model_config* m, const xc_gate_config* g, std::vector<int>& rows,
              std::vector<int>* grp_begin) {
  rows.clear();
  if (grp_begin) grp_begin->assign(1, 0);
  long long start = 0;
  std::vector<int> local;
  for (int gi = 0; gi < m->n_groups; ++gi) {
    const xc_view_group& vg = m->groups[gi];
    const long long T = (long long)vg.frames * vg.height * vg.width;
    camera_rows(vg, g->fp_budget, g->fp_mode, local);
    for (int v = 0; v < vg.views; ++v)
      for (int r : local) rows.push_back((int)(start + v * T + r));
    start += vg.views * T;
    if (grp_begin) grp_begin->push_back((int)rows.size());
  }
}

uint16_t f32_to_bf16_bits(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;  // NaN
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

struct Fail {
  xc_status s;
};

#define XC_HIP(call)                                  \
  do {                                                \
    hipError_t e_ = (call);                           \
    if (e_ != hipSuccess) throw Fail{XC_ERR_HIP};     \
  } while (0)

void* dalloc(xc_handle* h, size_t bytes) {
  if (bytes == 0) bytes = 256;
  void* p = nullptr;
  hipError_t e = hipMalloc(&p, bytes);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    throw Fail{e == hipErrorOutOfMemory ? XC_ERR_OOM : XC_ERR_HIP};
  }
  h->allocs.push_back(p);
  return p;
}

template <typename T>
T* dalloc_t(xc_handle* h, size_t count) {
  return reinterpret_cast<T*>(dalloc(h, count * sizeof(T)));
}

// Copy one float32 tensor of the host blob to its device slot, converting to
// bf16 when `to_bf16`.
void upload(xc_handle* h, const float* src, size_t count, void* dst, bool to_bf16, std::vector<uint16_t>& stage) {
  if (to_bf16) {
    stage.resize(count);
    for (size_t i = 0; i < count; ++i) stage[i] = f32_to_bf16_bits(src[i]);
    XC_HIP(hipMemcpyAsync(dst, stage.data(), count * 2, hipMemcpyHostToDevice, h->st));
  } else {
    XC_HIP(hipMemcpyAsync(dst, src, count * 4, hipMemcpyHostToDevice, h->st));
  }
  XC_HIP(hipStreamSynchronize(h->st));
}

// Kernel timing never fails a call: on any event error profiling switches off.
void prof_begin(xc_handle* h, int kind, ProfRecord* r) {
  r->start = r->stop = nullptr;
  if (!h->profiling || h->prof_suspended) return;
  hipEvent_t e[2];
  for (int i = 0; i < 2; ++i) {
    if (h->ev_free.empty()) {
      if (hipEventCreate(&e[i]) != hipSuccess) {
        (void)hipGetLastError();
        h->profiling = false;
        if (i == 1) h->ev_free.push_back(e[0]);
        return;
      }
    } else {
      e[i] = h->ev_free.back();
      h->ev_free.pop_back();
    }
  }
  r->kind = kind;
  r->start = e[0];
  r->stop = e[1];
  if (hipEventRecord(r->start, h->st) != hipSuccess) {
    (void)hipGetLastError();
    h->profiling = false;
    h->ev_free.push_back(e[0]);
    h->ev_free.push_back(e[1]);
    r->start = r->stop = nullptr;
  }
}

void prof_end(xc_handle* h, ProfRecord* r) {
  if (r->start == nullptr) return;
  if (hipEventRecord(r->stop, h->st) != hipSuccess) {
    (void)hipGetLastError();
    h->profiling = false;
    h->ev_free.push_back(r->start);
    h->ev_free.push_back(r->stop);
    return;
  }
  h->prof.push_back(*r);
}

struct Prof {
  xc_handle* h;
  ProfRecord r{};
  Prof(xc_handle* hh, int kind) : h(hh) { prof_begin(h, kind, &r); }
  ~Prof() { prof_end(h, &r); }
};

GateState gate_state(xc_handle* h) {
  GateState gs;
  gs.ema = h->ema;
  gs.stale = h->stale;
  gs.skip_counts = h->skip_counts;
  gs.flags = h->flags;
  gs.rec_dec = h->rec_dec;
  gs.rec_s = h->rec_s;
  gs.rec_d = h->rec_d;
  gs.rec_tau = h->rec_tau;
  gs.fp_sel = h->fp_sel;
  return gs;
}

PassWs own_ws(xc_handle* h) {
  PassWs ws;
  ws.records = h->fp_records;
  ws.attn = h->attn_ws;
  ws.attn_floats = h->attn_ws_floats;
  ws.prof = true;
  return ws;
}

template <typename P>
P* wptr(void* base, size_t elems_before, size_t esz) {
  return reinterpret_cast<P*>(reinterpret_cast<char*>(base) + elems_before * esz);
}

// Cross-attention layer of block b on x1 (in place): affine LayerNorm, q
// projection with the per-head RMSNorm, attention over the condition's keys
// and values, output projection added without a gate.
void cross_attention(xc_handle* h, int b, const int* flag, const PassWs& ws) {
  const int C = h->C, H = h->H, D = h->D;
  const int L = (int)h->L;
  const size_t esz = h->esz;
  const void* wq_c = wptr<void>(h->wqkv_c, (size_t)b * 3 * C * C, esz);
  {
    Prof p(h, XC_KERN_CROSS_Q);
    launch_ln_mod(h->dtype, h->x1, h->ln3_shift + (size_t)b * C, h->ln3_scale + (size_t)b * C, h->hbuf, L, C, flag,
                  h->st);
    EpiArgs e{};
    e.M = L;
    e.N = C;
    e.bias = h->bqkv_c + (size_t)b * 3 * C;
    if (h->dtype == XC_BF16) {
      e.gq = h->gq_c + (size_t)b * D;
      e.gk = h->gk_c + (size_t)b * D;
      e.q_out = h->q;
      e.H = H;
      e.D = D;
      e.Mpad = (int)h->Mpad;
      e.Lcap = (int)h->Lcap_c;
      launch_gemm(h->dtype, EPI_QKV, h->hbuf, wq_c, L, C, C, e, flag, h->st);
    } else {
      e.out_f32 = h->qkv;
      launch_gemm(h->dtype, EPI_BIAS_F32, h->hbuf, wq_c, L, C, C, e, flag, h->st);
      launch_qk_norm(h->dtype, h->qkv, nullptr, nullptr, C, h->gq_c + (size_t)b * D, h->gk_c + (size_t)b * D,
                     RopeArgs{}, h->q, nullptr, nullptr, L, H, D, (int)h->Mpad, 0, 0, flag, h->st);
    }
  }
  {
    Prof p(h, XC_KERN_CROSS_ATTENTION);
    launch_attention(h->dtype, h->q, wptr<void>(h->kc_c, (size_t)b * H * h->Lcap_c * D, esz),
                     wptr<void>(h->vt_c, (size_t)b * H * h->Lcap_c * D, esz), h->o, ws.attn, ws.attn_floats, L,
                     (int)h->Mpad,
                     (int)h->Lcap_c, h->n_cond, H, D, flag, h->st);
  }
  {
    Prof p(h, XC_KERN_CROSS_O);
    EpiArgs e{};
    e.M = L;
    e.N = C;
    e.bias = h->bo_c + (size_t)b * C;
    e.out_f32 = h->x1;
    e.resid = h->x1;  // each element is read and then written by the same lane
    e.gate = h->ones;
    launch_gemm(h->dtype, EPI_OPROJ, h->o, wptr<void>(h->wo_c, (size_t)b * C * C, esz), L, C, C, e, flag, h->st);
  }
}

// The compute sequence of block b (Eq. 1, the block of the DiT): LN+modulate,
// QKV projection, QK-norm and cache write, attention over the visible window,
// output projection with gated residual, LN+modulate, MLP up with GELU, MLP
// down with gated residual and (for gated blocks) the cached-residual store;
// models with a cross-attention layer run it between the output projection
// and the second LN+modulate.
// kv_only: stop after the key/value cache write (the block's output is not
// needed: the last block of a KV-update pass whose caller takes no output).
void compute_block(xc_handle* h, int b, const float* x, float* out, const int* flag, void* rhat_tb,
                   long long kv_off, long long Lk, const PassWs& ws, bool kv_only = false, bool col_sums = false) {
  const int C = h->C, H = h->H, D = h->D, Dm = h->Dm;
  const int L = (int)h->L;
  const size_t esz = h->esz;
  const float* mb = h->mod + (size_t)b * 6 * C;
  const float *shift1 = mb, *scale1 = mb + C, *gate1 = mb + 2 * C;
  const float *shift2 = mb + 3 * C, *scale2 = mb + 4 * C, *gate2 = mb + 5 * C;
  void* kc_b = wptr<void>(h->kc, (size_t)b * H * h->Lcap * D, esz);
  void* vt_b = wptr<void>(h->vt, (size_t)b * H * h->Lcap * D, esz);
  {
    // a skipped block's output x + rhat is written by this launch (Eq. 4)
    Prof p(h, flag ? XC_KERN_SKIP_ADD : XC_KERN_LN_MOD);
    launch_ln_mod(h->dtype, x, shift1, scale1, h->hbuf, L, C, flag, h->st, flag ? rhat_tb : nullptr,
                  flag ? out : nullptr);
  }
  if (h->dtype == XC_BF16) {
    // QKV projection with the per-head RMSNorm and the cache writes fused
    Prof p(h, XC_KERN_GEMM_QKV);
    EpiArgs e{};
    e.M = L;
    e.N = 3 * C;
    e.bias = h->bqkv + (size_t)b * 3 * C;
    e.gq = h->gq + (size_t)b * D;
    e.gk = h->gk + (size_t)b * D;
    e.q_out = h->q;
    e.k_cache = kc_b;
    e.vt_cache = vt_b;
    e.H = H;
    e.D = D;
    e.Mpad = (int)h->Mpad;
    e.Lcap = (int)h->Lcap;
    e.kv_off = (int)kv_off;
    e.rope = h->rope;
    launch_gemm(h->dtype, EPI_QKV, h->hbuf, wptr<void>(h->wqkv, (size_t)b * 3 * C * C, esz), L, 3 * C, C, e, flag,
                h->st);
  } else {
    {
      Prof p(h, XC_KERN_GEMM_QKV);
      EpiArgs e{};
      e.M = L;
      e.N = 3 * C;
      e.bias = h->bqkv + (size_t)b * 3 * C;
      e.out_f32 = h->qkv;
      launch_gemm(h->dtype, EPI_BIAS_F32, h->hbuf, wptr<void>(h->wqkv, (size_t)b * 3 * C * C, esz), L, 3 * C, C, e,
                  flag, h->st);
    }
    Prof p(h, XC_KERN_QK_NORM);
    launch_qk_norm(h->dtype, h->qkv, h->qkv + C, h->qkv + 2 * C, 3 * C, h->gq + (size_t)b * D,
                   h->gk + (size_t)b * D, h->rope, h->q, kc_b, vt_b, L, H, D, (int)h->Mpad, (int)h->Lcap,
                   (int)kv_off, flag, h->st);
  }
  if (kv_only) return;
  {
    Prof p(h, XC_KERN_ATTENTION);
    launch_attention(h->dtype, h->q, kc_b, vt_b, h->o, ws.attn, ws.attn_floats, L, (int)h->Mpad, (int)h->Lcap, (int)Lk,
                     H, D, flag, h->st);
  }
  {
    Prof p(h, XC_KERN_GEMM_OPROJ);
    EpiArgs e{};
    e.M = L;
    e.N = C;
    e.bias = h->bo + (size_t)b * C;
    e.out_f32 = h->x1;
    e.resid = x;
    e.gate = gate1;
    launch_gemm(h->dtype, EPI_OPROJ, h->o, wptr<void>(h->wo, (size_t)b * C * C, esz), L, C, C, e, flag, h->st);
  }
  if (h->Mc > 0) cross_attention(h, b, flag, ws);
  {
    Prof p(h, XC_KERN_LN_MOD);
    launch_ln_mod(h->dtype, h->x1, shift2, scale2, h->hbuf, L, C, flag, h->st);
  }
  {
    Prof p(h, XC_KERN_GEMM_UP);
    EpiArgs e{};
    e.M = L;
    e.N = Dm;
    e.bias = h->b1 + (size_t)b * Dm;
    e.out_t = h->u;
    launch_gemm(h->dtype, EPI_UP, h->hbuf, wptr<void>(h->w1, (size_t)b * Dm * C, esz), L, Dm, C, e, flag, h->st);
  }
  {
    Prof p(h, XC_KERN_GEMM_DOWN);
    EpiArgs e{};
    e.M = L;
    e.N = C;
    e.bias = h->b2 + (size_t)b * C;
    e.out_f32 = out;
    e.out_t = rhat_tb;
    e.resid = h->x1;
    e.gate = gate2;
    e.xin = x;
    if (col_sums && h->fold) {  // the next block's gate takes its global channel from these
      e.csum_part = h->csum_part;
      e.rb_split = h->rb_split;
      e.n_rb = h->n_rb;
    }
    launch_gemm(h->dtype, EPI_DOWN, h->u, wptr<void>(h->w2, (size_t)b * C * Dm, esz), L, C, Dm, e, flag, h->st);
  }
}

void pass_conditioning(xc_handle* h, float timestep, const float* action) {
  launch_cond(action, h->Dt, h->A, timestep, h->cond, h->st);
  Prof p(h, XC_KERN_ADALN);
  launch_adaln(h->dtype, h->w_ada, h->b_ada, h->cond, 6 * h->C, (long long)6 * h->C * h->Dc, h->B, h->Dc, h->mod,
               h->st);
}

xc_status check_launch() {
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? XC_OK : XC_ERR_HIP;
}

void build_tables(xc_handle* h) {
  const xc_model_config* m = &h->m;
  std::vector<int> cam_row_begin{0}, grp_cam_begin{0};
  long long start = 0;
  int cam = 0;
  for (int gi = 0; gi < m->n_groups; ++gi) {
    const xc_view_group& vg = m->groups[gi];
    const int T = vg.frames * vg.height * vg.width;
    for (int v = 0; v < vg.views; ++v, ++cam) {
      start += T;
      cam_row_begin.push_back((int)start);
    }
    grp_cam_begin.push_back(cam);
  }
  std::vector<int> rows, grp_srow_begin;
  all_rows(m, &h->g, rows, &grp_srow_begin);
  h->n_srows = (int)rows.size();
  h->n_cams = cam;
  h->fp_rows = h->n_srows + h->n_cams;
  h->spatial_count.assign(kMaxGroups, 1);
  for (int gi = 0; gi < m->n_groups; ++gi)
    h->spatial_count[gi] = (grp_srow_begin[gi + 1] - grp_srow_begin[gi]) * h->C;

  int* d_crb = dalloc_t<int>(h, cam_row_begin.size());
  int* d_gsb = dalloc_t<int>(h, grp_srow_begin.size());
  int* d_gcb = dalloc_t<int>(h, grp_cam_begin.size());
  int* d_rows = dalloc_t<int>(h, rows.size());
  XC_HIP(hipMemcpy(d_crb, cam_row_begin.data(), cam_row_begin.size() * 4, hipMemcpyHostToDevice));
  XC_HIP(hipMemcpy(d_gsb, grp_srow_begin.data(), grp_srow_begin.size() * 4, hipMemcpyHostToDevice));
  XC_HIP(hipMemcpy(d_gcb, grp_cam_begin.data(), grp_cam_begin.size() * 4, hipMemcpyHostToDevice));
  XC_HIP(hipMemcpy(d_rows, rows.data(), rows.size() * 4, hipMemcpyHostToDevice));
  FpTables& t = h->tables;
  t.n_cams = cam;
  t.cam_row_begin = d_crb;
  t.n_groups = m->n_groups;
  t.grp_srow_begin = d_gsb;
  t.grp_cam_begin = d_gcb;
  t.n_srows = h->n_srows;
  t.srows = d_rows;
  h->n_wg = gate_workgroups(h->C, h->n_srows, h->n_cams);
  h->fp_records = dalloc_t<double>(h, (size_t)h->n_wg * kMaxGroups * kFpRecord);

  // 32-row-block tables of the folded global channel: each block spans at
  // most two cameras when every camera has >= 32 tokens
  bool ok = h->g.enabled && h->dtype == XC_BF16;
  for (int v = 0; v < cam && ok; ++v) ok = cam_row_begin[v + 1] - cam_row_begin[v] >= 32;
  h->fold = ok;
  if (ok) {
    const int L = (int)h->L;
    h->n_rb = (L + 31) / 32;
    std::vector<int> rb_cam(h->n_rb), rb_split(h->n_rb, 32), lo(cam), hi(cam);
    for (int rb = 0, v = 0; rb < h->n_rb; ++rb) {
      while (cam_row_begin[v + 1] <= rb * 32) ++v;
      rb_cam[rb] = v;
      const int nxt = cam_row_begin[v + 1];
      if (v + 1 < cam && nxt < rb * 32 + 32) rb_split[rb] = nxt - rb * 32;
    }
    for (int v = 0; v < cam; ++v) {
      lo[v] = cam_row_begin[v] / 32;
      hi[v] = (cam_row_begin[v + 1] + 31) / 32;
    }
    h->rb_cam = dalloc_t<int>(h, h->n_rb);
    h->rb_split = dalloc_t<int>(h, h->n_rb);
    h->cam_rb_lo = dalloc_t<int>(h, cam);
    h->cam_rb_hi = dalloc_t<int>(h, cam);
    XC_HIP(hipMemcpy(h->rb_cam, rb_cam.data(), rb_cam.size() * 4, hipMemcpyHostToDevice));
    XC_HIP(hipMemcpy(h->rb_split, rb_split.data(), rb_split.size() * 4, hipMemcpyHostToDevice));
    XC_HIP(hipMemcpy(h->cam_rb_lo, lo.data(), lo.size() * 4, hipMemcpyHostToDevice));
    XC_HIP(hipMemcpy(h->cam_rb_hi, hi.data(), hi.size() * 4, hipMemcpyHostToDevice));
    h->csum_part = dalloc_t<float>(h, (size_t)2 * h->n_rb * 2 * h->C);
    h->csum_in = dalloc_t<double>(h, (size_t)h->B * cam * h->C);
    h->csum_rhat = dalloc_t<double>(h, (size_t)h->S * h->B * cam * h->C);
  }

}

// Rotary embedding: per-token packed (frame slot, h, w) and the table layout
// (frame slots, then rows 0..H_max-1, then columns 0..W_max-1).
void build_rope(xc_handle* h) {
  const xc_model_config* m = &h->m;
  std::vector<int> pos, slot_frames, slot_frame;
  int slot0 = 0, rows = 1, cols = 1;
  for (int gi = 0; gi < m->n_groups; ++gi) {
    const xc_view_group& vg = m->groups[gi];
    for (int v = 0; v < vg.views; ++v)
      for (int f = 0; f < vg.frames; ++f)
        for (int y = 0; y < vg.height; ++y)
          for (int x = 0; x < vg.width; ++x) pos.push_back((slot0 + f) | (y << 10) | (x << 20));
    for (int f = 0; f < vg.frames; ++f) {
      slot_frames.push_back(vg.frames);
      slot_frame.push_back(f);
    }
    slot0 += vg.frames;
    rows = std::max(rows, vg.height);
    cols = std::max(cols, vg.width);
  }
  const int s6 = h->D / 6;
  RopeArgs& r = h->rope;
  r.np[0] = (h->D - 4 * s6) / 2;
  r.np[1] = s6;
  r.np[2] = s6;
  r.off[0] = 0;
  r.off[1] = slot0 * r.np[0];
  r.off[2] = r.off[1] + rows * r.np[1];
  const int entries = r.off[2] + cols * r.np[2];
  h->rope_slots = slot0;
  h->rope_rows = rows;
  h->rope_cols = cols;
  h->rope_tab = dalloc_t<float2>(h, entries);
  h->rope_pos = dalloc_t<int>(h, pos.size());
  h->rope_slot_frames = dalloc_t<int>(h, slot_frames.size());
  h->rope_slot_frame = dalloc_t<int>(h, slot_frame.size());
  XC_HIP(hipMemcpy(h->rope_pos, pos.data(), pos.size() * 4, hipMemcpyHostToDevice));
  XC_HIP(hipMemcpy(h->rope_slot_frames, slot_frames.data(), slot_frames.size() * 4, hipMemcpyHostToDevice));
  XC_HIP(hipMemcpy(h->rope_slot_frame, slot_frame.data(), slot_frame.size() * 4, hipMemcpyHostToDevice));
  r.tab = h->rope_tab;
  r.pos = h->rope_pos;
}

// Frame positions follow the generation index: refill the tables for h->n.
void refresh_rope(xc_handle* h) {
  if (h->rope.tab == nullptr) return;
  launch_rope_table(h->rope_tab, h->rope, h->rope_slots, h->rope_slot_frames, h->rope_slot_frame, h->rope_rows,
                    h->rope_cols, (double)h->m.rope_theta, h->n, h->st);
}

void reset_state(xc_handle* h) {
  const size_t SB = (size_t)h->S * h->B;
  XC_HIP(hipMemsetAsync(h->kc, 0, (size_t)h->B * h->H * h->Lcap * h->D * h->esz, h->st));
  XC_HIP(hipMemsetAsync(h->vt, 0, (size_t)h->B * h->H * h->Lcap * h->D * h->esz, h->st));
  if (h->fp) XC_HIP(hipMemsetAsync(h->fp, 0, SB * h->fp_rows * h->C * sizeof(float), h->st));
  if (h->fp_alt) XC_HIP(hipMemsetAsync(h->fp_alt, 0, SB * h->fp_rows * h->C * sizeof(float), h->st));
  if (h->fp_sel) XC_HIP(hipMemsetAsync(h->fp_sel, 0, SB * sizeof(int), h->st));
  launch_fill_f32(h->ema, __builtin_nanf(""), (long long)SB, h->st);
  XC_HIP(hipMemsetAsync(h->stale, 0, SB * sizeof(int), h->st));
  XC_HIP(hipMemsetAsync(h->skip_counts, 0, SB * sizeof(int), h->st));
  XC_HIP(hipMemsetAsync(h->flags, 0, h->B * sizeof(int), h->st));
  XC_HIP(hipMemsetAsync(h->rec_dec, 0xff, h->B * sizeof(int), h->st));
  launch_fill_f32(h->rec_s, __builtin_nanf(""), h->B, h->st);
  launch_fill_f32(h->rec_d, __builtin_nanf(""), h->B, h->st);
  launch_fill_f32(h->rec_tau, __builtin_nanf(""), h->B, h->st);
  if (check_launch() != XC_OK) throw Fail{XC_ERR_HIP};
  h->n = 0;
  refresh_rope(h);
  if (check_launch() != XC_OK) throw Fail{XC_ERR_HIP};
  XC_HIP(hipStreamSynchronize(h->st));
  h->visited.assign(SB, 0);
  h->evals_post_warmup = h->gated_evals = h->kv_block_evals = 0;
  h->last_step = -1;
  h->any_forward = false;
  h->have_action_prev = false;
  h->have_action_cur = false;
}

void free_all(xc_handle* h) {
  for (void* p : h->allocs) (void)hipFree(p);
  h->allocs.clear();
  for (auto& r : h->prof) {
    (void)hipEventDestroy(r.start);
    (void)hipEventDestroy(r.stop);
  }
  h->prof.clear();
  for (hipEvent_t e : h->ev_free) (void)hipEventDestroy(e);
  h->ev_free.clear();
}

void init_device(xc_handle* h, const float* w) {
  const int B = h->B, C = h->C, D = h->D, Dm = h->Dm, Dc = h->Dc, S = h->S, H = h->H;
  const size_t esz = h->esz;
  const bool bf = h->dtype == XC_BF16;
  const size_t SB = (size_t)S * B;
  h->w_ada = dalloc(h, (size_t)B * 6 * C * Dc * esz);
  h->b_ada = dalloc_t<float>(h, (size_t)B * 6 * C);
  h->wqkv = dalloc(h, (size_t)B * 3 * C * C * esz);
  h->bqkv = dalloc_t<float>(h, (size_t)B * 3 * C);
  h->gq = dalloc_t<float>(h, (size_t)B * D);
  h->gk = dalloc_t<float>(h, (size_t)B * D);
  h->wo = dalloc(h, (size_t)B * C * C * esz);
  h->bo = dalloc_t<float>(h, (size_t)B * C);
  h->w1 = dalloc(h, (size_t)B * Dm * C * esz);
  h->b1 = dalloc_t<float>(h, (size_t)B * Dm);
  h->w2 = dalloc(h, (size_t)B * C * Dm * esz);
  h->b2 = dalloc_t<float>(h, (size_t)B * C);
  if (h->Mc > 0) {
    h->ln3_scale = dalloc_t<float>(h, (size_t)B * C);
    h->ln3_shift = dalloc_t<float>(h, (size_t)B * C);
    h->wqkv_c = dalloc(h, (size_t)B * 3 * C * C * esz);
    h->bqkv_c = dalloc_t<float>(h, (size_t)B * 3 * C);
    h->wo_c = dalloc(h, (size_t)B * C * C * esz);
    h->bo_c = dalloc_t<float>(h, (size_t)B * C);
    h->gq_c = dalloc_t<float>(h, (size_t)B * D);
    h->gk_c = dalloc_t<float>(h, (size_t)B * D);
  }

  // upload, block by block, in the blob order
  std::vector<uint16_t> stage;
  size_t off = 0;
  const size_t CC = (size_t)C * C;
  for (int b = 0; b < B; ++b) {
    upload(h, w + off, (size_t)6 * C * Dc, wptr<void>(h->w_ada, (size_t)b * 6 * C * Dc, esz), bf, stage);
    off += (size_t)6 * C * Dc;
    upload(h, w + off, (size_t)6 * C, h->b_ada + (size_t)b * 6 * C, false, stage);
    off += (size_t)6 * C;
    for (int part = 0; part < 3; ++part) {  // Wq, bq, Wk, bk, Wv, bv
      upload(h, w + off, CC, wptr<void>(h->wqkv, (size_t)b * 3 * CC + part * CC, esz), bf, stage);
      off += CC;
      upload(h, w + off, C, h->bqkv + (size_t)b * 3 * C + part * C, false, stage);
      off += C;
    }
    upload(h, w + off, CC, wptr<void>(h->wo, (size_t)b * CC, esz), bf, stage);
    off += CC;
    upload(h, w + off, C, h->bo + (size_t)b * C, false, stage);
    off += C;
    upload(h, w + off, (size_t)Dm * C, wptr<void>(h->w1, (size_t)b * Dm * C, esz), bf, stage);
    off += (size_t)Dm * C;
    upload(h, w + off, Dm, h->b1 + (size_t)b * Dm, false, stage);
    off += Dm;
    upload(h, w + off, (size_t)C * Dm, wptr<void>(h->w2, (size_t)b * C * Dm, esz), bf, stage);
    off += (size_t)C * Dm;
    upload(h, w + off, C, h->b2 + (size_t)b * C, false, stage);
    off += C;
    upload(h, w + off, D, h->gq + (size_t)b * D, false, stage);
    off += D;
    upload(h, w + off, D, h->gk + (size_t)b * D, false, stage);
    off += D;
    if (h->Mc > 0) {
      // LayerNorm scale w enters the modulated-LN kernel as 1 + (w - 1)
      std::vector<float> sc(w + off, w + off + C);
      for (float& v : sc) v -= 1.0f;
      upload(h, sc.data(), C, h->ln3_scale + (size_t)b * C, false, stage);
      off += C;
      upload(h, w + off, C, h->ln3_shift + (size_t)b * C, false, stage);
      off += C;
      for (int part = 0; part < 3; ++part) {  // Wq_c, bq_c, Wk_c, bk_c, Wv_c, bv_c
        upload(h, w + off, CC, wptr<void>(h->wqkv_c, (size_t)b * 3 * CC + part * CC, esz), bf, stage);
        off += CC;
        upload(h, w + off, C, h->bqkv_c + (size_t)b * 3 * C + part * C, false, stage);
        off += C;
      }
      upload(h, w + off, CC, wptr<void>(h->wo_c, (size_t)b * CC, esz), bf, stage);
      off += CC;
      upload(h, w + off, C, h->bo_c + (size_t)b * C, false, stage);
      off += C;
      upload(h, w + off, D, h->gq_c + (size_t)b * D, false, stage);
      off += D;
      upload(h, w + off, D, h->gk_c + (size_t)b * D, false, stage);
      off += D;
    }
  }

  h->kc = dalloc(h, (size_t)B * H * h->Lcap * D * esz);
  h->vt = dalloc(h, (size_t)B * H * h->Lcap * D * esz);
  if (h->g.enabled) {
    h->rhat = dalloc(h, SB * h->L * C * esz);
  }
  h->ema = dalloc_t<float>(h, SB);
  h->stale = dalloc_t<int>(h, SB);
  h->skip_counts = dalloc_t<int>(h, SB);
  h->flags = dalloc_t<int>(h, B);
  h->rec_dec = dalloc_t<int>(h, B);
  h->rec_s = dalloc_t<float>(h, B);
  h->rec_d = dalloc_t<float>(h, B);
  h->rec_tau = dalloc_t<float>(h, B);
  h->cond = dalloc_t<float>(h, kMaxCond);
  h->mod = dalloc_t<float>(h, (size_t)B * 6 * C);
  h->hbuf = dalloc(h, (size_t)h->Mpad * C * esz);
  if (!bf) h->qkv = dalloc_t<float>(h, (size_t)h->Mpad * 3 * C);
  h->q = dalloc(h, (size_t)H * h->Mpad * D * esz);
  h->o = dalloc(h, (size_t)h->Mpad * C * esz);
  h->u = dalloc(h, (size_t)h->Mpad * Dm * esz);
  h->x1 = dalloc_t<float>(h, (size_t)h->L * C);
  h->xa = dalloc_t<float>(h, (size_t)h->L * C);
  h->xb = dalloc_t<float>(h, (size_t)h->L * C);
  if (bf) {
    size_t ws = 0;  // the key window grows chunk by chunk: size for the largest need
    for (int w = 1; w <= h->Wkv; ++w) ws = std::max(ws, attention_workspace_floats((int)h->L, (int)(w * h->L), H, D));
    for (int n = 1; n <= h->Mc; ++n) ws = std::max(ws, attention_workspace_floats((int)h->L, n, H, D));
    if (ws) h->attn_ws = dalloc_t<float>(h, ws);
    h->attn_ws_floats = ws;
  }
  if (h->Mc > 0) {
    h->kc_c = dalloc(h, (size_t)B * H * h->Lcap_c * D * esz);
    h->vt_c = dalloc(h, (size_t)B * H * h->Lcap_c * D * esz);
    h->cond_act = dalloc(h, (size_t)h->Mcpad * C * esz);
    if (!bf) h->cond_kv = dalloc_t<float>(h, (size_t)h->Mcpad * 2 * C);
    h->ones = dalloc_t<float>(h, C);
    launch_fill_f32(h->ones, 1.0f, C, h->st);
    // keys past the valid condition tokens and padded token rows must be finite
    XC_HIP(hipMemsetAsync(h->kc_c, 0, (size_t)B * H * h->Lcap_c * D * esz, h->st));
    XC_HIP(hipMemsetAsync(h->vt_c, 0, (size_t)B * H * h->Lcap_c * D * esz, h->st));
    XC_HIP(hipMemsetAsync(h->cond_act, 0, (size_t)h->Mcpad * C * esz, h->st));
  }
  if (h->m.rope) build_rope(h);
  // padded activation rows are read by the tile loads and must be finite
  XC_HIP(hipMemsetAsync(h->hbuf, 0, (size_t)h->Mpad * C * esz, h->st));
  XC_HIP(hipMemsetAsync(h->q, 0, (size_t)H * h->Mpad * D * esz, h->st));
  XC_HIP(hipMemsetAsync(h->o, 0, (size_t)h->Mpad * C * esz, h->st));
  XC_HIP(hipMemsetAsync(h->u, 0, (size_t)h->Mpad * Dm * esz, h->st));
  build_tables(h);
  if (h->g.enabled) h->fp = dalloc_t<float>(h, SB * h->fp_rows * C);
  if (h->g.enabled && h->g.fp_refresh == XC_FP_REFRESH_ON_COMPUTE) {
    h->fp_alt = dalloc_t<float>(h, SB * h->fp_rows * C);
    h->fp_sel = dalloc_t<int>(h, SB);
  }
  reset_state(h);
}

GateArgs gate_args(xc_handle* h, int t, const float* action) {
  GateArgs ga{};
  ga.adaptive = h->g.adaptive;
  ga.tau_floor = h->g.tau_floor;
  ga.margin = h->g.margin;
  ga.alpha = h->g.alpha;
  ga.tau_cos_fixed = h->g.tau_cos_fixed;
  ga.tau_dev = h->g.tau_dev;
  ga.eps = h->g.eps;
  ga.max_stale = h->g.max_stale;
  ga.strict0 = (t == 0 && h->g.step0_mode == XC_STEP0_STRICT) ? 1 : 0;
  ga.tau_strict0 = h->g.tau_strict0;
  ga.n_groups = h->m.n_groups;
  ga.action_dim = h->have_action_prev ? h->A : 0;
  for (int i = 0; i < h->A; ++i) {
    ga.action[i] = action[i];
    ga.action_prev[i] = h->action_prev[i];
  }
  for (int gi = 0; gi < kMaxGroups; ++gi) ga.spatial_count[gi] = h->spatial_count[gi];
  return ga;
}

xc_status forward_pass(xc_handle* h, int32_t step, float timestep, const float* action_host, const void* x_in,
                       void* x_out, uint32_t flags, const PassWs& ws) {
  if (!h || !action_host || !x_in || !x_out) return XC_ERR_INVALID_ARG;
  if (h->sticky) return XC_ERR_HIP;
  if (h->Mc > 0 && h->n_cond == 0) return XC_ERR_STATE;
  if (step < 0 || step >= h->S) return XC_ERR_INVALID_ARG;
  if ((flags & ~(uint32_t)XC_FORCE_FULL) != 0) return XC_ERR_INVALID_ARG;
  if (!std::isfinite(timestep)) return XC_ERR_INVALID_ARG;
  for (int i = 0; i < h->A; ++i)
    if (!std::isfinite(action_host[i])) return XC_ERR_INVALID_ARG;
  if (action_changed(h, action_host)) return XC_ERR_STATE;
  h->prof_suspended = !ws.prof;
  try {
    XC_HIP(hipSetDevice(h->device));
    fix_action(h, action_host);
    const xc_gate_config& g = h->g;
    const bool forced_all = !g.enabled || h->n < g.warmup || (flags & XC_FORCE_FULL) ||
                            (step == 0 && g.step0_mode == XC_STEP0_FORCE);
    pass_conditioning(h, timestep, action_host);
    GateState gs = gate_state(h);
    launch_pass_begin(gs, h->B, h->st);
    const long long kv_off = (h->n % h->Wkv) * h->L;
    const long long Lk = std::min<long long>(h->n + 1, h->Wkv) * h->L;
    const GateArgs ga = gate_args(h, step, action_host);
    const float* x = reinterpret_cast<const float*>(x_in);
    for (int b = 0; b < h->B; ++b) {
      float* out = b == h->B - 1 ? reinterpret_cast<float*>(x_out) : ((b & 1) ? h->xb : h->xa);
      const int* flag = nullptr;
      void* rhat_tb = nullptr;
      if (gateable(h, b)) {
        const size_t sb = (size_t)step * h->B + b;
        rhat_tb = wptr<void>(h->rhat, sb * h->L * h->C, h->esz);
        const bool evaluate = !forced_all && h->visited[sb];
        {
          Prof p(h, XC_KERN_GATE);
          const size_t fo = sb * h->fp_rows * h->C;
          FoldArgs fa{};
          fa.full = (h->fold && b >= 1) ? 0 : 1;
          fa.b = b;
          fa.prev_gateable = b >= 1 && gateable(h, b - 1);
          fa.flags = h->flags;
          if (h->fold) {
            fa.csum_part = h->csum_part;
            fa.n_rb = h->n_rb;
            fa.cam_rb_lo = h->cam_rb_lo;
            fa.cam_rb_hi = h->cam_rb_hi;
            fa.rb_cam = h->rb_cam;
            fa.csum_in = h->csum_in;
            fa.csum_rhat = h->csum_rhat + (size_t)step * h->B * h->n_cams * h->C;
          }
          launch_fp_compare(x, h->C, h->tables, h->fp + fo, h->fp_alt ? h->fp_alt + fo : nullptr,
                            h->fp_sel ? h->fp_sel + sb : nullptr, ws.records, fa, h->st);
        }
        {
          Prof p(h, XC_KERN_GATE_DECIDE);
          launch_gate_decide(ws.records, h->n_wg, ga, gs, (int)sb, b, evaluate ? 1 : 0, h->st);
        }
        h->visited[sb] = 1;
        if (evaluate) {
          ++h->gated_evals;
          flag = h->flags + b;  // the block's first LayerNorm kernel also runs the skip path
        }
      }
      compute_block(h, b, x, out, flag, rhat_tb, kv_off, Lk, ws, false, b + 1 < h->B && gateable(h, b + 1));
      x = out;
    }
    if (h->n >= g.warmup) h->evals_post_warmup += h->B;
    h->last_step = step;
    h->any_forward = true;
    if (check_launch() != XC_OK) throw Fail{XC_ERR_HIP};
  } catch (const Fail& f) {
    h->prof_suspended = false;
    if (f.s == XC_ERR_HIP) h->sticky = true;
    return f.s;
  }
  h->prof_suspended = false;
  return XC_OK;
}

}  // namespace

extern "C" {

const char* xc_status_string(xc_status s) {
  switch (s) {
    case XC_OK: return "XC_OK";
    case XC_ERR_INVALID_ARG: return "XC_ERR_INVALID_ARG";
    case XC_ERR_STATE: return "XC_ERR_STATE";
    case XC_ERR_OOM: return "XC_ERR_OOM";
    case XC_ERR_HIP: return "XC_ERR_HIP";
    case XC_ERR_UNSUPPORTED: return "XC_ERR_UNSUPPORTED";
  }
  return "XC_ERR_UNKNOWN";
}

xc_status xc_init(const xc_model_config* model, const xc_gate_config* gate, const float* weights_host,
                  size_t weights_bytes, void* hip_stream, xc_handle** out) {
  if (!out || !weights_host) return XC_ERR_INVALID_ARG;
  xc_status s = validate_model(model);
  if (s != XC_OK) return s;
  s = validate_gate(gate, model);
  if (s != XC_OK) return s;
  const long long C = model->hidden, Dc = model->temb_dim + model->action_dim, Dm = model->mlp_hidden;
  const long long per_block = 6 * C * Dc + 6 * C + 4 * (C * C + C) + 2 * Dm * C + Dm + C + 2 * model->head_dim +
                              (model->cond_len > 0 ? 2 * C + 4 * (C * C + C) + 2 * model->head_dim : 0);
  if (weights_bytes != (size_t)(per_block * model->n_blocks) * sizeof(float)) return XC_ERR_INVALID_ARG;

  xc_handle* h = new (std::nothrow) xc_handle();
  if (!h) return XC_ERR_OOM;
  h->m = *model;
  h->g = *gate;
  h->st = (hipStream_t)hip_stream;
  h->B = model->n_blocks;
  h->C = model->hidden;
  h->H = model->n_heads;
  h->D = model->head_dim;
  h->Dm = model->mlp_hidden;
  h->Dt = model->temb_dim;
  h->A = model->action_dim;
  h->Dc = (int)Dc;
  h->S = model->n_steps;
  h->Wkv = model->kv_window;
  h->dtype = model->dtype;
  h->esz = model->dtype == XC_BF16 ? 2 : 4;
  h->L = tokens_of(model);
  // activation rows padded for every GEMM tile height (128, 192, 256) and the
  // 256-query attention tiles: roundup(L, 256) + 256 >= roundup(L, 192)
  h->Mpad = (h->L + 255) / 256 * 256 + 256;
  h->Lcap = ((long long)h->Wkv * h->L + 63) / 64 * 64;
  h->Mc = model->cond_len;
  h->Mcpad = ((long long)h->Mc + 255) / 256 * 256 + 256;
  h->Lcap_c = ((long long)h->Mc + 63) / 64 * 64;
  try {
    XC_HIP(hipGetDevice(&h->device));
    // null if the lookup failed: xc_forward_chunk_noalloc then returns XC_ERR_STATE
    h->scratch = device_scratch(h->device);
    init_device(h, weights_host);
  } catch (const Fail& f) {
    (void)hipGetLastError();
    free_all(h);
    delete h;
    return f.s;
  } catch (const std::bad_alloc&) {
    free_all(h);
    delete h;
    return XC_ERR_OOM;
  }
  *out = h;
  return XC_OK;
}

xc_status xc_forward_chunk(xc_handle* h, int32_t step, float timestep, const float* action_host, const void* x_in,
                           void* x_out, uint32_t flags) {
  if (!h) return XC_ERR_INVALID_ARG;
  return forward_pass(h, step, timestep, action_host, x_in, x_out, flags, own_ws(h));
}

xc_status xc_forward_chunk_noalloc(xc_handle* h, int32_t step, float timestep, const float* action_host,
                                   const void* x_in, void* x_out, uint32_t flags) {
  if (!h) return XC_ERR_INVALID_ARG;
  if (h->scratch == nullptr) return XC_ERR_STATE;
  // the gate's records first, the attention partials in the rest (256-byte aligned)
  const size_t rec_bytes = ((size_t)h->n_wg * kMaxGroups * kFpRecord * sizeof(double) + 255) / 256 * 256;
  if (rec_bytes > kStaticScratchBytes) return XC_ERR_UNSUPPORTED;
  PassWs ws;
  ws.records = reinterpret_cast<double*>(h->scratch);
  ws.attn = reinterpret_cast<float*>(h->scratch + rec_bytes);
  ws.attn_floats = (kStaticScratchBytes - rec_bytes) / sizeof(float);
  ws.prof = false;
  return forward_pass(h, step, timestep, action_host, x_in, x_out, flags, ws);
}

xc_status xc_kv_update(xc_handle* h, float timestep, const float* action_host, const void* x_clean, void* x_out) {
  if (!h || !action_host || !x_clean) return XC_ERR_INVALID_ARG;
  if (h->sticky) return XC_ERR_HIP;
  if (h->Mc > 0 && h->n_cond == 0) return XC_ERR_STATE;
  if (!std::isfinite(timestep)) return XC_ERR_INVALID_ARG;
  for (int i = 0; i < h->A; ++i)
    if (!std::isfinite(action_host[i])) return XC_ERR_INVALID_ARG;
  if (action_changed(h, action_host)) return XC_ERR_STATE;
  try {
    XC_HIP(hipSetDevice(h->device));
    pass_conditioning(h, timestep, action_host);
    const long long kv_off = (h->n % h->Wkv) * h->L;
    const long long Lk = std::min<long long>(h->n + 1, h->Wkv) * h->L;
    const float* x = reinterpret_cast<const float*>(x_clean);
    for (int b = 0; b < h->B; ++b) {
      float* out = (b & 1) ? h->xb : h->xa;
      if (b == h->B - 1 && x_out) out = reinterpret_cast<float*>(x_out);
      compute_block(h, b, x, out, nullptr, nullptr, kv_off, Lk, own_ws(h), b == h->B - 1 && !x_out);
      x = out;
    }
    h->kv_block_evals += h->B;
    for (int i = 0; i < h->A; ++i) h->action_prev[i] = action_host[i];
    h->have_action_prev = true;
    h->have_action_cur = false;
    h->n += 1;
    refresh_rope(h);
    h->last_step = h->S;
    if (check_launch() != XC_OK) throw Fail{XC_ERR_HIP};
  } catch (const Fail& f) {
    if (f.s == XC_ERR_HIP) h->sticky = true;
    return f.s;
  }
  return XC_OK;
}

xc_status xc_set_condition(xc_handle* h, const float* cond_host, int32_t n_tokens) {
  if (!h || !cond_host) return XC_ERR_INVALID_ARG;
  if (h->sticky) return XC_ERR_HIP;
  if (h->Mc == 0) return XC_ERR_STATE;
  if (n_tokens < 1 || n_tokens > h->Mc) return XC_ERR_INVALID_ARG;
  const int C = h->C, H = h->H, D = h->D;
  const size_t count = (size_t)n_tokens * C;
  for (size_t i = 0; i < count; ++i)
    if (!std::isfinite(cond_host[i])) return XC_ERR_INVALID_ARG;
  try {
    XC_HIP(hipSetDevice(h->device));
    const bool bf = h->dtype == XC_BF16;
    const size_t esz = h->esz;
    std::vector<uint16_t> stage;
    upload(h, cond_host, count, h->cond_act, bf, stage);
    // each block's K_c = RMSNorm(Wk_c cond + bk_c) * gk_c and V_c = Wv_c cond + bv_c
    for (int b = 0; b < h->B; ++b) {
      const void* wkv = wptr<void>(h->wqkv_c, (size_t)b * 3 * C * C + (size_t)C * C, esz);
      void* kc_b = wptr<void>(h->kc_c, (size_t)b * H * h->Lcap_c * D, esz);
      void* vt_b = wptr<void>(h->vt_c, (size_t)b * H * h->Lcap_c * D, esz);
      EpiArgs e{};
      e.M = n_tokens;
      e.N = 2 * C;
      e.bias = h->bqkv_c + (size_t)b * 3 * C + C;
      if (bf) {
        e.part_base = 1;
        e.gq = h->gq_c + (size_t)b * D;
        e.gk = h->gk_c + (size_t)b * D;
        e.k_cache = kc_b;
        e.vt_cache = vt_b;
        e.H = H;
        e.D = D;
        e.Mpad = (int)h->Mcpad;
        e.Lcap = (int)h->Lcap_c;
        launch_gemm(h->dtype, EPI_QKV, h->cond_act, wkv, n_tokens, 2 * C, C, e, nullptr, h->st);
      } else {
        e.out_f32 = h->cond_kv;
        launch_gemm(h->dtype, EPI_BIAS_F32, h->cond_act, wkv, n_tokens, 2 * C, C, e, nullptr, h->st);
        launch_qk_norm(h->dtype, nullptr, h->cond_kv, h->cond_kv + C, 2 * C, h->gq_c + (size_t)b * D,
                       h->gk_c + (size_t)b * D, RopeArgs{}, nullptr, kc_b, vt_b, n_tokens, H, D, 0,
                       (int)h->Lcap_c, 0, nullptr, h->st);
      }
    }
    if (check_launch() != XC_OK) throw Fail{XC_ERR_HIP};
    XC_HIP(hipStreamSynchronize(h->st));
    h->n_cond = n_tokens;
  } catch (const Fail& f) {
    h->sticky = true;
    return f.s;
  }
  return XC_OK;
}

xc_status xc_stats(xc_handle* h, xc_stats_t* stats, int32_t* skip_counts, uint8_t* last_decision, float* last_cos,
                   float* last_dev, float* last_tau, float* ema) {
  if (!h) return XC_ERR_INVALID_ARG;
  if (h->sticky) return XC_ERR_HIP;
  try {
    XC_HIP(hipSetDevice(h->device));
    XC_HIP(hipStreamSynchronize(h->st));
    const size_t SB = (size_t)h->S * h->B;
    std::vector<int> counts(SB);
    XC_HIP(hipMemcpy(counts.data(), h->skip_counts, SB * sizeof(int), hipMemcpyDeviceToHost));
    if (stats) {
      long long skips = 0;
      for (int c : counts) skips += c;
      stats->generations = h->n;
      stats->evals_post_warmup = h->evals_post_warmup;
      stats->gated_evals = h->gated_evals;
      stats->skips = skips;
      stats->kv_block_evals = h->kv_block_evals;
      stats->last_step = h->last_step;
    }
    if (skip_counts) std::memcpy(skip_counts, counts.data(), SB * sizeof(int));
    if (last_decision) {
      std::vector<int> dec(h->B);
      XC_HIP(hipMemcpy(dec.data(), h->rec_dec, h->B * sizeof(int), hipMemcpyDeviceToHost));
      for (int b = 0; b < h->B; ++b) last_decision[b] = h->any_forward ? (uint8_t)dec[b] : (uint8_t)XC_DEC_NONE;
    }
    if (last_cos) XC_HIP(hipMemcpy(last_cos, h->rec_s, h->B * sizeof(float), hipMemcpyDeviceToHost));
    if (last_dev) XC_HIP(hipMemcpy(last_dev, h->rec_d, h->B * sizeof(float), hipMemcpyDeviceToHost));
    if (last_tau) XC_HIP(hipMemcpy(last_tau, h->rec_tau, h->B * sizeof(float), hipMemcpyDeviceToHost));
    if (ema) XC_HIP(hipMemcpy(ema, h->ema, SB * sizeof(float), hipMemcpyDeviceToHost));
  } catch (const Fail& f) {
    h->sticky = true;
    return f.s;
  }
  return XC_OK;
}

xc_status xc_read_cache(xc_handle* h, int32_t kind, int32_t step, int32_t block, void* out_dev, size_t out_floats) {
  if (!h || !out_dev) return XC_ERR_INVALID_ARG;
  if (h->sticky) return XC_ERR_HIP;
  if (block < 0 || block >= h->B) return XC_ERR_INVALID_ARG;
  if (kind == XC_CACHE_RESIDUAL) {
    if (step < 0 || step >= h->S) return XC_ERR_INVALID_ARG;
    if (!gateable(h, block) || h->rhat == nullptr) return XC_ERR_STATE;
    if (out_floats != (size_t)h->L * h->C) return XC_ERR_INVALID_ARG;
  } else if (kind == XC_CACHE_KEYS || kind == XC_CACHE_VALUES) {
    if (out_floats != (size_t)h->H * h->Wkv * h->L * h->D) return XC_ERR_INVALID_ARG;
  } else {
    return XC_ERR_INVALID_ARG;
  }
  try {
    XC_HIP(hipSetDevice(h->device));
    float* out = reinterpret_cast<float*>(out_dev);
    if (kind == XC_CACHE_RESIDUAL) {
      const size_t sb = (size_t)step * h->B + block;
      launch_read_cache(h->dtype, wptr<void>(h->rhat, sb * h->L * h->C, h->esz), out, 1, (int)h->L, h->C, h->L, 0,
                        h->st);
    } else {
      const void* src = wptr<void>(kind == XC_CACHE_KEYS ? h->kc : h->vt, (size_t)block * h->H * h->Lcap * h->D, h->esz);
      launch_read_cache(h->dtype, src, out, h->H, (int)(h->Wkv * h->L), h->D, h->Lcap, kind == XC_CACHE_VALUES ? 1 : 0,
                        h->st);
    }
    if (check_launch() != XC_OK) throw Fail{XC_ERR_HIP};
  } catch (const Fail& f) {
    h->sticky = true;
    return f.s;
  }
  return XC_OK;
}

xc_status xc_reset(xc_handle* h) {
  if (!h) return XC_ERR_INVALID_ARG;
  if (h->sticky) return XC_ERR_HIP;
  try {
    XC_HIP(hipSetDevice(h->device));
    reset_state(h);
  } catch (const Fail& f) {
    h->sticky = true;
    return f.s;
  }
  return XC_OK;
}

xc_status xc_destroy(xc_handle* h) {
  if (!h) return XC_OK;
  (void)hipSetDevice(h->device);
  (void)hipStreamSynchronize(h->st);
  free_all(h);
  delete h;
  return XC_OK;
}

xc_status xc_axpby(xc_handle* h, float a, const void* x, float b, const void* y, void* out, size_t n) {
  if (!h || !x || !y || !out) return XC_ERR_INVALID_ARG;
  if (h->sticky) return XC_ERR_HIP;
  if (n == 0) return XC_OK;
  (void)hipSetDevice(h->device);
  launch_axpby(a, reinterpret_cast<const float*>(x), b, reinterpret_cast<const float*>(y),
               reinterpret_cast<float*>(out), (long long)n, h->st);
  if (check_launch() != XC_OK) {
    h->sticky = true;
    return XC_ERR_HIP;
  }
  return XC_OK;
}

xc_status xc_fingerprint_rows(const xc_model_config* model, const xc_gate_config* gate, int32_t* rows, size_t cap,
                              size_t* n_rows) {
  if (!n_rows) return XC_ERR_INVALID_ARG;
  xc_status s = validate_model(model);
  if (s != XC_OK) return s;
  s = validate_gate(gate, model);
  if (s != XC_OK) return s;
  std::vector<int> all;
  all_rows(model, gate, all, nullptr);
  *n_rows = all.size();
  if (rows)
    for (size_t i = 0; i < all.size() && i < cap; ++i) rows[i] = all[i];
  return XC_OK;
}

xc_status xc_mfma_rate(int32_t shape, int32_t random_operands, void* stream, double* tflops) {
  if (!tflops || shape < 0 || shape > 4) return XC_ERR_INVALID_ARG;
  *tflops = 0.0;
  return mfma_rate(shape, random_operands != 0, reinterpret_cast<hipStream_t>(stream), tflops) == hipSuccess
             ? XC_OK
             : XC_ERR_HIP;
}

xc_status xc_lds_dma_rate(int32_t row_bytes, void* stream, double* tbytes_per_s) {
  if (!tbytes_per_s || (row_bytes != 64 && row_bytes != 128 && row_bytes != 256)) return XC_ERR_INVALID_ARG;
  *tbytes_per_s = 0.0;
  const hipError_t e = lds_dma_rate(row_bytes, reinterpret_cast<hipStream_t>(stream), tbytes_per_s);
  if (e == hipErrorOutOfMemory) return XC_ERR_OOM;
  return e == hipSuccess ? XC_OK : XC_ERR_HIP;
}

xc_status xc_profile(xc_handle* h, int32_t enable) {
  if (!h) return XC_ERR_INVALID_ARG;
  h->profiling = enable != 0;
  return XC_OK;
}

xc_status xc_kernel_times(xc_handle* h, int32_t kind, int64_t* launches, double* total_ms, int32_t clear) {
  if (!h || kind < 0 || kind >= XC_KERN_COUNT) return XC_ERR_INVALID_ARG;
  if (h->sticky) return XC_ERR_HIP;
  try {
    XC_HIP(hipSetDevice(h->device));
    XC_HIP(hipStreamSynchronize(h->st));
    long long cnt = 0;
    double tot = 0.0;
    std::vector<ProfRecord> keep;
    for (const ProfRecord& r : h->prof) {
      if (r.kind != kind) {
        keep.push_back(r);
        continue;
      }
      float ms = 0.f;
      XC_HIP(hipEventElapsedTime(&ms, r.start, r.stop));
      ++cnt;
      tot += ms;
      if (clear) {
        h->ev_free.push_back(r.start);
        h->ev_free.push_back(r.stop);
      } else {
        keep.push_back(r);
      }
    }
    h->prof.swap(keep);
    if (launches) *launches = cnt;
    if (total_ms) *total_ms = tot;
  } catch (const Fail& f) {
    h->sticky = true;
    return f.s;
  }
  return XC_OK;
}

}  // extern "C"
