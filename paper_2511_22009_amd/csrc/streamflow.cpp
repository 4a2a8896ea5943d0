// C-ABI runtime of the stream-batched rectified-flow step: blob parsing and
// validation, weight upload, workspace, and the launch sequence of one
// heterogeneous-timestep network call (Sec. 3.2, Eq. 5) followed by the per-sample
// Euler update and queue shift (Alg. 1's final update; Alg. 2). Every computation
// runs in the HIP kernels of this library; this file only validates and enqueues.
#include "streamflow.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstddef>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <new>
#include <vector>

#include "sf_launch.h"

namespace sf {

FastDiv make_fastdiv(uint32_t d) {
  FastDiv f;
  f.d = d;
  uint32_t s = 0;
  while ((1ull << s) < d) ++s;
  f.shift = s;
  f.magic = (uint32_t)((((1ull << 32) * ((1ull << s) - d)) / d) + 1);
  return f;
}

}  // namespace sf

thread_local sf::LaunchEvents sf::t_launch_events{nullptr, nullptr};

namespace {

constexpr size_t kAlign = 256;
constexpr int kTimingPool = 4096;

struct Header {
  char magic[4];
  uint32_t version;
  uint32_t C, H, W, p, D, L, heads, mlp, tdim, ctx_len, ctx_dim, has_cross;
  uint64_t seed;
};
static_assert(sizeof(Header) == 64, "blob header is 64 bytes");

struct Block {
  void *W_qkv, *W_o, *W_fc1, *W_fc2, *W_qx, *W_kvx, *W_ox;
  float *b_qkv, *b_o, *b_fc1, *b_fc2, *b_qx, *b_kvx, *b_ox;
};

struct Timing {
  bool on = false;
  std::vector<hipEvent_t> ev;  // start/end pairs
  int used = 0;
  long launches = 0;
};

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// Bump allocator over one device allocation: first pass sizes, second pass assigns.
struct Carver {
  char* base = nullptr;
  size_t off = 0;
  template <typename T>
  T* take(size_t count, size_t elem = sizeof(T)) {
    T* p = (T*)(base ? base + off : nullptr);
    off = align_up(off + count * elem);
    return p;
  }
};

uint16_t f32_to_bf16(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);  // quiet NaN
  u += 0x7fffu + ((u >> 16) & 1u);                                            // round to nearest even
  return (uint16_t)(u >> 16);
}

}  // namespace

struct sf_model {
  Header hd{};
  int N = 0, P = 0, dh = 0, modw = 0, E = 0;
  int prec = SF_PREC_BF16;
  bool bf16 = true;
  int max_rows = 0;
  size_t es = 2;  // bytes per compute-type element
  char* wmem = nullptr;
  size_t wbytes = 0;
  char* wsmem = nullptr;
  size_t wsbytes = 0;
  // weights
  float *W_pe = nullptr, *b_pe = nullptr, *pos = nullptr, *W_t1 = nullptr, *b_t1 = nullptr;
  float *W_t2 = nullptr, *b_t2 = nullptr, *freqs = nullptr, *b_mod = nullptr, *W_f = nullptr, *b_f = nullptr;
  void* W_mod = nullptr;  // [modw][D], every block's projection then the final layer's
  std::vector<Block> blk;
  // workspace
  float *hid = nullptr, *svec = nullptr, *table = nullptr, *h = nullptr, *vrows = nullptr;
  // the fixed scratch array of sf_modulation_noalloc on this model's device
  float* scratch = nullptr;
  size_t scratch_floats = 0;
  void *act = nullptr, *q = nullptr, *k = nullptr, *vT = nullptr, *o = nullptr, *f = nullptr;
  // cross-attention context entries: n_entries contexts (fp32 copy and GEMM operand),
  // their keys [n_entries][L][heads][ctx_len][dh] and transposed values
  // [n_entries][L][heads][dh][ldvx] for every block, and the entries' device state
  void *ctxA = nullptr, *kx = nullptr, *vTx = nullptr;
  float* ctx_keep = nullptr;
  sf::CtxState* ctx_st = nullptr;
  int n_entries = 0;
  int ctx_lp = 0;  // context tokens per entry in ctxA and kx: ctx_len rounded up to 16 (zero rows)
  bool ctx_cache_on = false;
  // every block's context K/V projection, contiguous: [L][2D][ctx_dim] and [L][2D]
  void* W_kvx = nullptr;
  float* b_kvx = nullptr;
  int ldv = 0, ldvx = 0;
  int vperm = 0;  // transposed v in the permuted key layout (vt_pos): bf16 mode
  Timing timing[SF_KC_COUNT];
  // graph replay: captured launch sequences keyed by the call's arguments
  struct GraphEntry {
    std::vector<char> key;
    hipGraphExec_t exec = nullptr;
    unsigned long long used = 0;
  };
  // PeRFlow time windows (windows == 0: Euler on the velocity)
  int windows = 0;
  double win_eps = 0.0;
  double* abar = nullptr;
  int n_abar = 0;
  bool graph_on = false;
  std::vector<GraphEntry> graphs;
  unsigned long long graph_clock = 0;
  long graph_replays = 0;
  // modulation cache: the timesteps (and stream) the adaLN table rows were last
  // computed for, so a call with the same timesteps can skip the conditioning launches
  bool mod_cache_on = false;
  bool mod_valid = false;
  int mod_n = 0;
  float mod_t[SF_MAX_ROWS] = {};
  hipStream_t mod_stream = nullptr;
  long mod_skips = 0;
};

namespace {

// ---------------------------------------------------------------- validation
int check_header(const void* blob, size_t nbytes, Header* out, size_t* expect) {
  if (nbytes < sizeof(Header)) return SF_E_BLOB;
  Header h;
  std::memcpy(&h, blob, sizeof(Header));
  if (std::memcmp(h.magic, "SFW1", 4) != 0 || h.version != 1) return SF_E_BLOB;
  const uint32_t dims[] = {h.C, h.H, h.W, h.p, h.D, h.heads, h.mlp, h.tdim};
  for (uint32_t d : dims)
    if (d == 0 || d > 65536) return SF_E_BLOB;
  if (h.L > 4096 || h.has_cross > 1 || h.ctx_len > 65536 || h.ctx_dim > 65536) return SF_E_BLOB;
  if (h.has_cross && (h.ctx_len == 0 || h.ctx_dim == 0)) return SF_E_BLOB;
  if (h.H % h.p || h.W % h.p || h.D % h.heads || h.tdim % 2) return SF_E_BLOB;
  const uint64_t D = h.D, P = (uint64_t)h.p * h.p * h.C, F = h.mlp;
  const uint64_t N = (uint64_t)(h.H / h.p) * (h.W / h.p);
  uint64_t floats = D * P + D + N * D + D * h.tdim + D + D * D + D;
  uint64_t per_block = 6 * D * D + 6 * D + 3 * D * D + 3 * D + D * D + D + F * D + F + D * F + D;
  if (h.has_cross) per_block += D * D + D + 2 * D * h.ctx_dim + 2 * D + D * D + D;
  floats += per_block * h.L + 2 * D * D + 2 * D + P * D + P;
  *expect = sizeof(Header) + 4 * floats;
  if (nbytes != *expect) return SF_E_BLOB;
  *out = h;
  return SF_OK;
}

int check_supported(const Header& h) {
  const uint32_t P = h.p * h.p * h.C;
  const uint32_t dh = h.D / h.heads;
  if (h.D % 8 || h.D > (uint32_t)sf::kMaxWidth || h.mlp % 8 || h.tdim % 8 ||
      h.tdim > (uint32_t)sf::kMaxWidth || P > (uint32_t)sf::kMaxPatch || !sf::attention_supports((int)dh) ||
      (h.C * h.H * h.W) % 4 || (h.has_cross && h.ctx_dim % 8))
    return SF_E_UNSUPPORTED;
  return SF_OK;
}

// The bf16 GEMMs and attention address their operands through buffer resources with
// 32-bit byte offsets (int arithmetic, kOffOOB as the past-the-end sentinel), so every
// activation operand must stay below kOffOOB bytes at the loaded row count; the fp32
// kernels index with size_t and are bounded only by the element counts.
int check_capacity(const Header& h, int max_rows, size_t es) {
  const uint64_t N = (uint64_t)(h.H / h.p) * (h.W / h.p);
  const uint64_t R = (uint64_t)max_rows;
  const uint64_t widest = h.mlp > h.D ? h.mlp : h.D;
  const uint64_t limit = es == 2 ? (uint64_t)sf::kOffOOBHost : (1ull << 31);
  const uint64_t unit = es == 2 ? es : 1;  // bytes (bf16) or elements (fp32)
  if (R * N * widest * unit >= limit) return SF_E_UNSUPPORTED;
  // cross-attention: the context entries (max_rows + 1) and every block's K/V weights,
  // the operands of one GEMM
  const uint64_t ctx_lp = ((uint64_t)h.ctx_len + 15) / 16 * 16;
  if (h.has_cross && ((R + 1) * ctx_lp * (uint64_t)(h.ctx_dim > h.D ? h.ctx_dim : h.D) * unit >= limit ||
                      (uint64_t)h.L * 2 * h.D * h.ctx_dim * unit >= limit))
    return SF_E_UNSUPPORTED;
  return SF_OK;
}

bool finite_all(const float* a, int n) {
  for (int i = 0; i < n; ++i)
    if (!std::isfinite(a[i])) return false;
  return true;
}

// ------------------------------------------------------------------ layout
// Sizes (pass 1, base == nullptr) or assigns (pass 2) every weight pointer.
void carve_weights(sf_model* m, Carver& cv) {
  const Header& h = m->hd;
  const size_t D = h.D, P = m->P, F = h.mlp;
  m->W_pe = cv.take<float>(D * P);
  m->b_pe = cv.take<float>(D);
  m->pos = cv.take<float>((size_t)m->N * D);
  m->W_t1 = cv.take<float>(D * h.tdim);
  m->b_t1 = cv.take<float>(D);
  m->W_t2 = cv.take<float>(D * D);
  m->b_t2 = cv.take<float>(D);
  m->freqs = cv.take<float>(h.tdim / 2);
  m->W_mod = cv.take<char>((size_t)m->modw * D, m->es);
  m->b_mod = cv.take<float>(m->modw);
  m->blk.resize(h.L);
  if (h.has_cross) {
    m->W_kvx = cv.take<char>((size_t)h.L * 2 * D * h.ctx_dim, m->es);
    m->b_kvx = cv.take<float>((size_t)h.L * 2 * D);
  }
  for (uint32_t l = 0; l < h.L; ++l) {
    Block& b = m->blk[l];
    b.W_qkv = cv.take<char>(3 * D * D, m->es);
    b.b_qkv = cv.take<float>(3 * D);
    b.W_o = cv.take<char>(D * D, m->es);
    b.b_o = cv.take<float>(D);
    if (h.has_cross) {
      b.W_qx = cv.take<char>(D * D, m->es);
      b.b_qx = cv.take<float>(D);
      b.W_kvx = m->W_kvx ? (char*)m->W_kvx + (size_t)l * 2 * D * h.ctx_dim * m->es : nullptr;
      b.b_kvx = m->b_kvx ? m->b_kvx + (size_t)l * 2 * D : nullptr;
      b.W_ox = cv.take<char>(D * D, m->es);
      b.b_ox = cv.take<float>(D);
    } else {
      b.W_qx = b.W_kvx = b.W_ox = nullptr;
      b.b_qx = b.b_kvx = b.b_ox = nullptr;
    }
    b.W_fc1 = cv.take<char>(F * D, m->es);
    b.b_fc1 = cv.take<float>(F);
    b.W_fc2 = cv.take<char>(D * F, m->es);
    b.b_fc2 = cv.take<float>(D);
  }
  m->W_f = cv.take<float>(P * D);
  m->b_f = cv.take<float>(P);
}

void carve_workspace(sf_model* m, Carver& cv) {
  const Header& h = m->hd;
  const size_t R = m->max_rows, D = h.D, N = m->N, M = R * N;
  m->hid = cv.take<float>(R * D);
  m->svec = cv.take<float>(R * D);
  m->table = cv.take<float>(R * m->modw);
  m->h = cv.take<float>(M * D);
  m->vrows = cv.take<float>(R * m->E);
  m->act = cv.take<char>(M * D, m->es);
  m->q = cv.take<char>(M * D, m->es);
  m->k = cv.take<char>(M * D, m->es);
  m->vT = cv.take<char>(R * D * m->ldv, m->es);
  m->o = cv.take<char>(M * D, m->es);
  m->f = cv.take<char>(M * h.mlp, m->es);
  if (h.has_cross) {
    const size_t NE = m->n_entries, per_row = (size_t)h.ctx_len * h.ctx_dim;
    m->ctxA = cv.take<char>(NE * m->ctx_lp * h.ctx_dim, m->es);
    m->ctx_keep = cv.take<float>(NE * per_row);
    m->kx = cv.take<char>(NE * h.L * m->ctx_lp * D, m->es);
    m->vTx = cv.take<char>(NE * h.L * D * m->ldvx, m->es);
    m->ctx_st = cv.take<sf::CtxState>(1);
  }
}

// Host image of the device weight region, filled from the blob in blob order.
void fill_weights(sf_model* m, const char* blob, std::vector<char>& img) {
  const Header& h = m->hd;
  const size_t D = h.D, P = m->P, F = h.mlp;
  const float* src = (const float*)(blob + sizeof(Header));
  char* base = img.data();
  auto dev_off = [&](const void* p) { return (size_t)((const char*)p - m->wmem); };
  auto put_f32 = [&](const void* dst, size_t n) {
    std::memcpy(base + dev_off(dst), src, n * 4);
    src += n;
  };
  auto put_w = [&](const void* dst, size_t n, size_t elem_off = 0) {
    char* d = base + dev_off(dst) + elem_off * m->es;
    if (m->bf16) {
      uint16_t* o = (uint16_t*)d;
      for (size_t i = 0; i < n; ++i) o[i] = f32_to_bf16(src[i]);
    } else {
      std::memcpy(d, src, n * 4);
    }
    src += n;
  };
  {  // W_pe [D][P] in the blob, stored transposed [P][D] for coalesced reads
    float* dst = (float*)(base + dev_off(m->W_pe));
    for (size_t d = 0; d < D; ++d)
      for (size_t f = 0; f < P; ++f) dst[f * D + d] = src[d * P + f];
    src += D * P;
  }
  put_f32(m->b_pe, D);
  put_f32(m->pos, (size_t)m->N * D);
  put_f32(m->W_t1, D * h.tdim);
  put_f32(m->b_t1, D);
  put_f32(m->W_t2, D * D);
  put_f32(m->b_t2, D);
  for (uint32_t l = 0; l < h.L; ++l) {
    const Block& b = m->blk[l];
    put_w(m->W_mod, 6 * D * D, (size_t)l * 6 * D * D);
    std::memcpy(base + dev_off(m->b_mod) + (size_t)l * 6 * D * 4, src, 6 * D * 4);
    src += 6 * D;
    put_w(b.W_qkv, 3 * D * D);
    put_f32(b.b_qkv, 3 * D);
    put_w(b.W_o, D * D);
    put_f32(b.b_o, D);
    if (h.has_cross) {
      put_w(b.W_qx, D * D);
      put_f32(b.b_qx, D);
      put_w(b.W_kvx, 2 * D * h.ctx_dim);
      put_f32(b.b_kvx, 2 * D);
      put_w(b.W_ox, D * D);
      put_f32(b.b_ox, D);
    }
    put_w(b.W_fc1, F * D);
    put_f32(b.b_fc1, F);
    put_w(b.W_fc2, D * F);
    put_f32(b.b_fc2, D);
  }
  put_w(m->W_mod, 2 * D * D, (size_t)h.L * 6 * D * D);
  std::memcpy(base + dev_off(m->b_mod) + (size_t)h.L * 6 * D * 4, src, 2 * D * 4);
  src += 2 * D;
  put_f32(m->W_f, P * D);
  put_f32(m->b_f, P);
  // sinusoid frequencies 10000^(-i/half), evaluated in double and rounded once
  float* fq = (float*)(base + dev_off(m->freqs));
  const int half = h.tdim / 2;
  for (int i = 0; i < half; ++i) fq[i] = (float)std::exp(-std::log(10000.0) * (double)i / (double)half);
}

// ------------------------------------------------------------- launch helpers
// Classes whose launch is one kernel get the events on that kernel's own dispatch
// (pure kernel time); the others (several kernels) are bracketed on the stream.
constexpr bool one_kernel_class(int kc) { return kc != SF_KC_TEMB && kc != SF_KC_CROSS; }

template <typename F>
int timed(sf_model* m, int kc, hipStream_t s, F&& launch) {
  Timing& tm = m->timing[kc];
  const bool rec = tm.on && tm.used < kTimingPool;
  hipEvent_t e0 = rec ? tm.ev[2 * tm.used] : nullptr, e1 = rec ? tm.ev[2 * tm.used + 1] : nullptr;
  const bool attach = rec && one_kernel_class(kc);
  if (rec && !attach && hipEventRecord(e0, s) != hipSuccess) return SF_E_HIP;
  if (attach) sf::t_launch_events = sf::LaunchEvents{e0, e1};
  const hipError_t err = launch();
  const bool consumed = attach && sf::t_launch_events.start == nullptr;
  sf::t_launch_events = sf::LaunchEvents{nullptr, nullptr};
  if (err != hipSuccess) return SF_E_HIP;
  if (tm.on) ++tm.launches;
  if (rec) {
    if (attach && !consumed && hipEventRecord(e0, s) != hipSuccess) return SF_E_HIP;  // nothing launched
    if ((!attach || !consumed) && hipEventRecord(e1, s) != hipSuccess) return SF_E_HIP;
    ++tm.used;
  }
  return SF_OK;
}

#define SF_TRY(x)                 \
  do {                            \
    int rc_ = (x);                \
    if (rc_ != SF_OK) return rc_; \
  } while (0)

// Per-sample conditioning: t[k] -> adaLN table row k (width modw). hid and svec hold the
// timestep MLP's hidden layer and SiLU(c) ([n][D] each). With `embed`, the patch embed
// runs in the same launch as the adaLN projections where that kernel supports it, and
// *embedded says whether it did.
int run_modulation(sf_model* m, const float* t, int n, float* table, hipStream_t s, float* hid, float* svec,
                   const sf::EmbedArgs* embed = nullptr, bool* embedded = nullptr) {
  const Header& h = m->hd;
  return timed(m, SF_KC_TEMB, s, [&]() -> hipError_t {
    sf::GemvArgs g{};
    g.W = m->W_t1;
    g.bias = m->b_t1;
    g.B = n;
    g.K = h.tdim;
    g.R = h.D;
    g.Y = hid;
    g.ldy = h.D;
    g.act = 1;
    g.x_mode = 1;
    g.freqs = m->freqs;
    for (int i = 0; i < n; ++i) g.t.v[i] = t[i];
    hipError_t e = sf::launch_gemv(false, g, s);
    if (e != hipSuccess) return e;
    sf::GemvArgs g2{};
    g2.W = m->W_t2;
    g2.bias = m->b_t2;
    g2.X = hid;
    g2.ldx = h.D;
    g2.B = n;
    g2.K = h.D;
    g2.R = h.D;
    g2.Y = svec;
    g2.ldy = h.D;
    g2.act = 1;  // the adaLN projections read SiLU(c)
    e = sf::launch_gemv(false, g2, s);
    if (e != hipSuccess) return e;
    sf::GemvArgs g3{};
    g3.W = m->W_mod;
    g3.bias = m->b_mod;
    g3.X = svec;
    g3.ldx = h.D;
    g3.B = n;
    g3.K = h.D;
    g3.R = m->modw;
    g3.Y = table;
    g3.ldy = m->modw;
    if (embed && sf::gemv_embed_supported(m->bf16, g3, *embed)) {
      *embedded = true;
      return sf::launch_gemv_embed(m->bf16, g3, *embed, s);
    }
    return sf::launch_gemv(m->bf16, g3, s);
  });
}

bool any_timing(const sf_model* m) {
  for (const Timing& tm : m->timing)
    if (tm.on) return true;
  return false;
}

sf::GemmArgs gemm_base(const void* A, int lda, const void* B, int ldb, int M, int N, int K, const float* bias) {
  sf::GemmArgs g{};
  g.A = A;
  g.lda = lda;
  g.B = B;
  g.ldb = ldb;
  g.M = M;
  g.N = N;
  g.K = K;
  g.bias = bias;
  return g;
}

// The network call on `rows` rows built from n_lat latents (rows = n_lat, or 2 n_lat
// with guidance: cond rows then uncond rows, each using its latent's t). Runs through
// `nblocks` blocks; if head_out != nullptr also the output head into head_out [rows][E].
int run_network(sf_model* m, const float* x, const float* t, int n_lat, int rows, const sf_cond* cond,
                int nblocks, float* head_out, hipStream_t s, bool table_ready = false) {
  const Header& h = m->hd;
  const int D = h.D, N = m->N, M = rows * N;
  const sf::EmbedArgs emb{x, n_lat, m->W_pe, m->b_pe, m->pos, m->h, rows, (int)h.C, (int)h.H, (int)h.W, (int)h.p, D, N};
  // the embed shares the adaLN projections' launch unless per-class times are taken
  bool embedded = false;
  if (!table_ready)
    SF_TRY(run_modulation(m, t, n_lat, m->table, s, m->hid, m->svec, any_timing(m) ? nullptr : &emb, &embedded));
  if (!embedded) SF_TRY(timed(m, SF_KC_EMBED, s, [&]() { return sf::launch_embed(emb, s); }));
  const sf::FastDiv div_n = sf::make_fastdiv(N), div_d = sf::make_fastdiv(D), div_dh = sf::make_fastdiv(m->dh);
  const sf::FastDiv div_ctx = sf::make_fastdiv(h.has_cross ? m->ctx_lp : 1);
  const int* kv_map = nullptr;
  if (h.has_cross) {
    // the context entries of this call (reused or assembled), then the keys and values
    // of every block for them in one GEMM; entries that are reused skip their tiles
    const bool guided = rows > n_lat;
    const sf::CtxArgs c{cond->ctx, guided ? cond->null_ctx : nullptr, n_lat, guided ? 1 : 0,
                        (int)(h.ctx_len * h.ctx_dim), m->n_entries, m->ctx_keep, m->ctxA,
                        (int)(m->ctx_lp * h.ctx_dim), m->ctx_st};
    const char* st = (const char*)m->ctx_st;
    kv_map = (const int*)(st + offsetof(sf::CtxState, kv_map));
    SF_TRY(timed(m, SF_KC_CROSS, s, [&]() -> hipError_t {
      const hipError_t e = m->ctx_cache_on ? sf::launch_ctx_lookup(m->bf16, c, s) : sf::launch_ctx_prepare(m->bf16, c, s);
      if (e != hipSuccess) return e;
      const int entries = m->ctx_cache_on ? m->n_entries : n_lat + (guided ? 1 : 0);
      sf::GemmArgs g = gemm_base(m->ctxA, h.ctx_dim, m->W_kvx, h.ctx_dim, entries * m->ctx_lp, 2 * D * h.L, h.ctx_dim,
                                 m->b_kvx);
      g.k = m->kx; g.vT = m->vTx; g.heads = h.heads; g.dh = m->dh; g.D = D; g.ntok = m->ctx_lp;
      g.ldv = m->ldvx; g.which_base = 1; g.vperm = m->vperm; g.kv_blocks = h.L;
      g.div_ntok = div_ctx; g.div_D = div_d; g.div_dh = div_dh;
      g.row_live = m->ctx_cache_on ? (const int*)(st + offsetof(sf::CtxState, live)) : nullptr;
      return sf::launch_gemm(m->bf16, sf::EPI_KVX, g, s);
    }));
  }
  auto ln = [&](int shift_off, int scale_off, bool modulate) {
    sf::LnArgs a{m->h, m->act, M, D, modulate ? m->table : nullptr, m->modw, shift_off, scale_off, div_n, n_lat};
    return sf::launch_ln(m->bf16, a, s);
  };
  for (int l = 0; l < nblocks; ++l) {
    const Block& b = m->blk[l];
    const int base = l * 6 * D;
    SF_TRY(timed(m, SF_KC_LN, s, [&]() { return ln(base, base + D, true); }));
    SF_TRY(timed(m, SF_KC_QKV, s, [&]() {
      sf::GemmArgs g = gemm_base(m->act, D, b.W_qkv, D, M, 3 * D, D, b.b_qkv);
      g.q = m->q; g.k = m->k; g.vT = m->vT;
      g.heads = h.heads; g.dh = m->dh; g.D = D; g.ntok = N; g.ldv = m->ldv; g.which_base = 0; g.vperm = m->vperm;
      g.div_ntok = div_n; g.div_D = div_d; g.div_dh = div_dh;
      return sf::launch_gemm(m->bf16, sf::EPI_QKV, g, s);
    }));
    SF_TRY(timed(m, SF_KC_ATTN, s, [&]() {
      sf::AttnArgs a{m->q, m->k, m->vT, m->o, rows, (int)h.heads, N, N, m->dh, m->ldv, D,
                     (float)(1.0 / std::sqrt((double)m->dh)), m->vperm};
      return sf::launch_attention(m->bf16, a, s);
    }));
    SF_TRY(timed(m, SF_KC_PROJ, s, [&]() {
      sf::GemmArgs g = gemm_base(m->o, D, b.W_o, D, M, D, D, b.b_o);
      g.h = m->h; g.ldh = D; g.table = m->table; g.ldt = m->modw; g.gate_off = base + 2 * D;
      g.n_slots = n_lat; g.div_ntok = div_n;
      return sf::launch_gemm(m->bf16, sf::EPI_RES_GATE, g, s);
    }));
    if (h.has_cross) {
      SF_TRY(timed(m, SF_KC_CROSS, s, [&]() -> hipError_t {
        hipError_t e = ln(0, 0, false);
        if (e != hipSuccess) return e;
        sf::GemmArgs gq = gemm_base(m->act, D, b.W_qx, D, M, D, D, b.b_qx);
        gq.q = m->q; gq.heads = h.heads; gq.dh = m->dh; gq.D = D; gq.ntok = N; gq.which_base = 0; gq.vperm = m->vperm;
        gq.div_ntok = div_n; gq.div_D = div_d; gq.div_dh = div_dh;
        if ((e = sf::launch_gemm(m->bf16, sf::EPI_QKV, gq, s)) != hipSuccess) return e;
        // row r reads entry kv_map[r], block l of it (ctx_len keys of ctx_lp rows per head)
        const size_t kblk = (size_t)h.heads * m->ctx_lp * m->dh, vblk = (size_t)h.heads * m->dh * m->ldvx;
        sf::AttnArgs a{m->q, (const char*)m->kx + l * kblk * m->es, (const char*)m->vTx + l * vblk * m->es, m->o,
                       rows, (int)h.heads, N, (int)h.ctx_len, m->dh, m->ldvx, D,
                       (float)(1.0 / std::sqrt((double)m->dh)), m->vperm};
        a.kv_map = kv_map;
        a.k_ld = m->ctx_lp;
        a.k_rs = h.L * kblk;
        a.v_rs = h.L * vblk;
        if ((e = sf::launch_attention(m->bf16, a, s)) != hipSuccess) return e;
        sf::GemmArgs go = gemm_base(m->o, D, b.W_ox, D, M, D, D, b.b_ox);
        go.h = m->h; go.ldh = D;
        return sf::launch_gemm(m->bf16, sf::EPI_RES, go, s);
      }));
    }
    SF_TRY(timed(m, SF_KC_LN, s, [&]() { return ln(base + 3 * D, base + 4 * D, true); }));
    SF_TRY(timed(m, SF_KC_FC1, s, [&]() {
      sf::GemmArgs g = gemm_base(m->act, D, b.W_fc1, D, M, h.mlp, D, b.b_fc1);
      g.out = m->f; g.ldo = h.mlp;
      return sf::launch_gemm(m->bf16, sf::EPI_GELU, g, s);
    }));
    SF_TRY(timed(m, SF_KC_FC2, s, [&]() {
      sf::GemmArgs g = gemm_base(m->f, h.mlp, b.W_fc2, h.mlp, M, D, h.mlp, b.b_fc2);
      g.h = m->h; g.ldh = D; g.table = m->table; g.ldt = m->modw; g.gate_off = base + 5 * D;
      g.n_slots = n_lat; g.div_ntok = div_n;
      return sf::launch_gemm(m->bf16, sf::EPI_RES_GATE_MLP, g, s);
    }));
  }
  if (!head_out) return SF_OK;
  return timed(m, SF_KC_HEAD, s, [&]() {
    sf::HeadArgs a{};
    a.h = m->h; a.W_f = m->W_f; a.b_f = m->b_f; a.table = m->table; a.ldt = m->modw;
    a.shift_off = (int)h.L * 6 * D; a.scale_off = (int)h.L * 6 * D + D; a.n_slots = n_lat; a.tok = div_n;
    a.v = head_out; a.rows = rows; a.C = h.C; a.H = h.H; a.W = h.W; a.p = h.p; a.D = D; a.N = N; a.P = m->P;
    return sf::launch_head(a, s);
  });
}

// Validates the call-side conditioning and returns the network row count (0 = invalid).
int rows_for(const sf_model* m, int B, const sf_cond* cond, bool* guided, float* w) {
  *guided = false;
  *w = 0.0f;
  if (m->hd.has_cross) {
    if (!cond || !cond->ctx) return 0;
    if (cond->null_ctx) {
      if (!std::isfinite(cond->guidance)) return 0;
      *guided = true;
      *w = cond->guidance;
    }
  } else if (cond) {
    return 0;
  }
  const int rows = *guided ? 2 * B : B;
  return (B >= 1 && rows <= m->max_rows) ? rows : 0;
}

int fail_alloc_after() {
  const char* e = std::getenv("SF_FAIL_ALLOC_AFTER");
  return e ? std::atoi(e) : -1;
}

// Copies the model's time-window scheduler (if any) and the slots' times into the
// update's arguments.
void set_windows(const sf_model* m, const float* t, int B, sf::EulerArgs& a) {
  a.windows = m->windows;
  a.eps = m->win_eps;
  a.abar = m->abar;
  a.n_abar = m->n_abar;
  for (int i = 0; i < B; ++i) a.t.v[i] = t[i];
}

// ---------------------------------------------------------------- modulation cache
// True when the cache is on and the adaLN table already holds the rows of exactly these
// timesteps (bitwise), computed by an earlier call on the same stream: the call can then
// skip the conditioning launches (the table depends on t only).
bool modulation_cached(const sf_model* m, const float* t, int n, hipStream_t s) {
  return m->mod_cache_on && m->mod_valid && m->mod_n == n && m->mod_stream == s &&
         std::memcmp(m->mod_t, t, sizeof(float) * n) == 0;
}

// Records what a network call left in the table: the rows of t[0..n) if it computed them
// (or reused them) and succeeded; nothing valid otherwise.
int note_modulation(sf_model* m, const float* t, int n, hipStream_t s, int rc) {
  // a failed call may have left the context entries half updated: forget them
  if (rc != SF_OK && m->ctx_cache_on && m->ctx_st) (void)sf::launch_ctx_reset(m->ctx_st, s);
  m->mod_valid = rc == SF_OK;
  if (m->mod_valid) {
    m->mod_n = n;
    std::memcpy(m->mod_t, t, sizeof(float) * n);
    m->mod_stream = s;
  }
  return rc;
}

// ---------------------------------------------------------------- graph replay
constexpr size_t kMaxGraphs = 64;

template <typename T>
void key_put(std::vector<char>& k, const T& v) {
  const char* p = reinterpret_cast<const char*>(&v);
  k.insert(k.end(), p, p + sizeof(T));
}

std::vector<char> call_key(const sf_model* m, int kind, const void* a, const void* b, const void* c, const void* d, int B,
                           const float* t, const float* dt, const sf_cond* cond, hipStream_t s,
                           bool table_ready) {
  std::vector<char> k;
  key_put(k, kind);
  key_put(k, table_ready);
  key_put(k, a);
  key_put(k, b);
  key_put(k, c);
  key_put(k, d);
  key_put(k, B);
  key_put(k, (const void*)s);
  for (int i = 0; i < B; ++i) key_put(k, t[i]);
  if (dt)
    for (int i = 0; i < B; ++i) key_put(k, dt[i]);
  const bool has = cond != nullptr;
  key_put(k, has);
  key_put(k, m->ctx_cache_on);
  if (has) {
    key_put(k, (const void*)cond->ctx);
    key_put(k, (const void*)cond->null_ctx);
    key_put(k, cond->guidance);
  }
  return k;
}

void drop_graphs(sf_model* m) {
  for (auto& g : m->graphs)
    if (g.exec) (void)hipGraphExecDestroy(g.exec);
  m->graphs.clear();
}

// Runs `enqueue` (which launches the call's kernels on s) through the graph cache: a
// cached graph for `key` is replayed; otherwise the launches are captured, instantiated,
// cached and replayed. Eager when graphs are off, on the null stream, or while timing.
template <typename F>
int run_graphed(sf_model* m, const std::vector<char>& key, hipStream_t s, F&& enqueue) {
  if (!m->graph_on || s == nullptr || any_timing(m)) return enqueue();
  for (auto& g : m->graphs) {
    if (g.key == key) {
      g.used = ++m->graph_clock;
      ++m->graph_replays;
      return hipGraphLaunch(g.exec, s) == hipSuccess ? SF_OK : SF_E_HIP;
    }
  }
  if (hipStreamBeginCapture(s, hipStreamCaptureModeThreadLocal) != hipSuccess) return SF_E_HIP;
  const int rc = enqueue();
  hipGraph_t graph = nullptr;
  const hipError_t ec = hipStreamEndCapture(s, &graph);
  if (rc != SF_OK || ec != hipSuccess || !graph) {
    if (graph) (void)hipGraphDestroy(graph);
    return rc != SF_OK ? rc : SF_E_HIP;
  }
  hipGraphExec_t exec = nullptr;
  const hipError_t ei = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
  (void)hipGraphDestroy(graph);
  if (ei != hipSuccess || !exec) return SF_E_HIP;
  if (m->graphs.size() >= kMaxGraphs) {
    auto lru = m->graphs.begin();
    for (auto it = m->graphs.begin(); it != m->graphs.end(); ++it)
      if (it->used < lru->used) lru = it;
    (void)hipGraphExecDestroy(lru->exec);
    m->graphs.erase(lru);
  }
  sf_model::GraphEntry e;
  e.key = key;
  e.exec = exec;
  e.used = ++m->graph_clock;
  m->graphs.push_back(std::move(e));
  return hipGraphLaunch(exec, s) == hipSuccess ? SF_OK : SF_E_HIP;
}

}  // namespace

extern "C" {

const char* sf_strerror(int code) {
  switch (code) {
    case SF_OK: return "ok";
    case SF_E_INVAL: return "invalid argument";
    case SF_E_BLOB: return "malformed weight blob";
    case SF_E_NOTLOADED: return "model not loaded";
    case SF_E_OOM: return "device allocation failed";
    case SF_E_HIP: return "HIP runtime or kernel launch error";
    case SF_E_UNSUPPORTED: return "shape not supported by this build";
    default: return "unknown status code";
  }
}

int sf_load_weights(const void* blob, size_t nbytes, int precision, int max_rows, sf_model** out) {
  if (!blob || !out) return SF_E_INVAL;
  *out = nullptr;
  if (precision != SF_PREC_BF16 && precision != SF_PREC_FP32) return SF_E_INVAL;
  if (max_rows < 1 || max_rows > SF_MAX_ROWS) return SF_E_INVAL;
  Header h;
  size_t expect = 0;
  int rc = check_header(blob, nbytes, &h, &expect);
  if (rc != SF_OK) return rc;
  if ((rc = check_supported(h)) != SF_OK) return rc;
  if ((rc = check_capacity(h, max_rows, precision == SF_PREC_BF16 ? 2 : 4)) != SF_OK) return rc;

  sf_model* m = new (std::nothrow) sf_model();
  if (!m) return SF_E_OOM;
  m->hd = h;
  m->N = (int)((h.H / h.p) * (h.W / h.p));
  m->P = (int)(h.p * h.p * h.C);
  m->dh = (int)(h.D / h.heads);
  m->modw = (int)(h.L * 6 * h.D + 2 * h.D);
  m->E = (int)(h.C * h.H * h.W);
  m->prec = precision;
  m->bf16 = precision == SF_PREC_BF16;
  m->es = m->bf16 ? 2 : 4;
  m->max_rows = max_rows;
  // transposed v: rows padded to whole 64-key steps of the attention kernels (the
  // permuted layout moves keys within a group of 16, and the head-dim-64 kernel loads
  // whole steps without a column check); columns of no key stay zero from the
  // workspace clear
  m->ldv = (m->N + 63) / 64 * 64;
  m->ldvx = h.has_cross ? (int)((h.ctx_len + 63) / 64 * 64) : 0;
  // one entry per conditional row plus the null context (a call has at most max_rows
  // context rows and one null row)
  m->n_entries = h.has_cross ? max_rows + 1 : 0;
  // a context entry spans whole 16-token groups, so the transposed values of every
  // 16 tokens leave the projection's epilogue as vector stores
  m->ctx_lp = h.has_cross ? (int)((h.ctx_len + 15) / 16 * 16) : 0;
  m->vperm = m->bf16 ? 1 : 0;

  Carver cw;
  carve_weights(m, cw);
  m->wbytes = cw.off;
  Carver cs;
  carve_workspace(m, cs);
  m->wsbytes = cs.off;

  const int fail_after = fail_alloc_after();
  int allocs = 0;
  auto dev_alloc = [&](char** p, size_t n) -> int {
    if (fail_after >= 0 && allocs++ >= fail_after) return SF_E_OOM;
    if (hipMalloc((void**)p, n) != hipSuccess) {
      *p = nullptr;
      (void)hipGetLastError();
      return SF_E_OOM;
    }
    return SF_OK;
  };
  if ((rc = dev_alloc(&m->wmem, m->wbytes)) != SF_OK || (rc = dev_alloc(&m->wsmem, m->wsbytes)) != SF_OK) {
    sf_free(m);
    return rc;
  }
  Carver cw2;
  cw2.base = m->wmem;
  carve_weights(m, cw2);
  Carver cs2;
  cs2.base = m->wsmem;
  carve_workspace(m, cs2);

  std::vector<char> img;
  try {
    img.assign(m->wbytes, 0);
  } catch (...) {
    sf_free(m);
    return SF_E_OOM;
  }
  // set-up of the allocation-free conditioning call: the device address of the fixed
  // scratch array on this (current) device, looked up once per device
  if (sf::modulation_scratch(&m->scratch, &m->scratch_floats) != hipSuccess) {
    (void)hipGetLastError();
    sf_free(m);
    return SF_E_HIP;
  }
  fill_weights(m, (const char*)blob, img);
  if (hipMemcpy(m->wmem, img.data(), m->wbytes, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemset(m->wsmem, 0, m->wsbytes) != hipSuccess || hipDeviceSynchronize() != hipSuccess) {
    sf_free(m);
    return SF_E_HIP;
  }
  *out = m;
  return SF_OK;
}

void sf_free(sf_model* m) {
  if (!m) return;
  if (m->wmem || m->wsmem) (void)hipDeviceSynchronize();
  drop_graphs(m);
  if (m->abar) (void)hipFree(m->abar);
  for (auto& tm : m->timing)
    for (hipEvent_t e : tm.ev) (void)hipEventDestroy(e);
  if (m->wmem) (void)hipFree(m->wmem);
  if (m->wsmem) (void)hipFree(m->wsmem);
  delete m;
}

int sf_get_info(const sf_model* m, sf_info* info) {
  if (!m) return SF_E_NOTLOADED;
  if (!info) return SF_E_INVAL;
  const Header& h = m->hd;
  info->C = h.C; info->H = h.H; info->W = h.W; info->p = h.p; info->D = h.D; info->L = h.L;
  info->heads = h.heads; info->mlp = h.mlp; info->tdim = h.tdim; info->ctx_len = h.ctx_len;
  info->ctx_dim = h.ctx_dim; info->has_cross = h.has_cross; info->tokens = m->N; info->mod_width = m->modw;
  info->precision = m->prec; info->max_rows = m->max_rows; info->weight_bytes = m->wbytes;
  info->workspace_bytes = m->wsbytes;
  info->vt_ld = m->ldv;
  info->vt_key_perm = m->vperm;
  return SF_OK;
}

int sf_velocity(sf_model* m, const float* x, const float* t, int B, const sf_cond* cond, float* v, void* stream) {
  if (!m) return SF_E_NOTLOADED;
  if (!x || !t || !v || B < 1 || B > SF_MAX_ROWS || !finite_all(t, B)) return SF_E_INVAL;
  bool guided;
  float w;
  const int rows = rows_for(m, B, cond, &guided, &w);
  if (!rows) return SF_E_INVAL;
  hipStream_t s = (hipStream_t)stream;
  const bool ready = modulation_cached(m, t, B, s);
  if (ready) ++m->mod_skips;
  const int rc = run_graphed(m, call_key(m, 0, x, v, nullptr, nullptr, B, t, nullptr, cond, s, ready), s, [&]() -> int {
    SF_TRY(run_network(m, x, t, B, rows, cond, m->hd.L, guided ? m->vrows : v, s, ready));
    if (guided) return timed(m, SF_KC_EULER, s, [&]() { return sf::launch_cfg_combine(m->vrows, B, m->E, w, v, s); });
    return SF_OK;
  });
  return note_modulation(m, t, B, s, rc);
}

int sf_stream_step(sf_model* m, float* x, const float* t, const float* dt, int B, const sf_cond* cond,
                   const float* z_new, float* x_done, void* stream) {
  if (!m) return SF_E_NOTLOADED;
  if (!x || !t || !dt || !z_new || B < 1 || B > SF_MAX_ROWS || !finite_all(t, B) || !finite_all(dt, B))
    return SF_E_INVAL;
  bool guided;
  float w;
  const int rows = rows_for(m, B, cond, &guided, &w);
  if (!rows) return SF_E_INVAL;
  hipStream_t s = (hipStream_t)stream;
  const bool ready = modulation_cached(m, t, B, s);
  if (ready) ++m->mod_skips;
  const int rc = run_graphed(m, call_key(m, 1, x, z_new, x_done, nullptr, B, t, dt, cond, s, ready), s, [&]() -> int {
    SF_TRY(run_network(m, x, t, B, rows, cond, m->hd.L, m->vrows, s, ready));
    return timed(m, SF_KC_EULER, s, [&]() {
      sf::EulerArgs a{};
      a.x = x; a.v = m->vrows; a.B = B; a.E = m->E; a.guided = guided ? 1 : 0; a.w = w;
      for (int i = 0; i < B; ++i) a.dt.v[i] = dt[i];
      a.z_new = z_new; a.x_done = x_done;
      set_windows(m, t, B, a);
      return sf::launch_euler_shift(a, s);
    });
  });
  return note_modulation(m, t, B, s, rc);
}

int sf_euler_shift(sf_model* m, float* x, const float* v, const float* dt, int B, const float* z_new,
                   float* x_done, void* stream) {
  if (!m) return SF_E_NOTLOADED;
  if (!x || !v || !dt || !z_new || B < 1 || B > SF_MAX_ROWS || !finite_all(dt, B)) return SF_E_INVAL;
  hipStream_t s = (hipStream_t)stream;
  return timed(m, SF_KC_EULER, s, [&]() {
    sf::EulerArgs a{};
    a.x = x; a.v = v; a.B = B; a.E = m->E; a.guided = 0; a.w = 0.0f;
    for (int i = 0; i < B; ++i) a.dt.v[i] = dt[i];
    a.z_new = z_new; a.x_done = x_done;
    return sf::launch_euler_shift(a, s);
  });
}

int sf_modulation(sf_model* m, const float* t, int B, float* table, void* stream) {
  if (!m) return SF_E_NOTLOADED;
  if (!t || !table || B < 1 || B > m->max_rows || !finite_all(t, B)) return SF_E_INVAL;
  return run_modulation(m, t, B, table, (hipStream_t)stream, m->hid, m->svec);
}

int sf_modulation_noalloc(sf_model* m, const float* t, int B, float* table, void* stream) {
  if (!m) return SF_E_NOTLOADED;
  if (!t || !table || B < 1 || B > SF_MAX_ROWS || !finite_all(t, B)) return SF_E_INVAL;
  // the two [B][D] intermediates must fit the fixed array (B <= 64 and D <= 2048 for
  // every loaded model, so this holds; checked all the same)
  if ((size_t)2 * B * m->hd.D > m->scratch_floats || !m->scratch) return SF_E_INVAL;
  float* hid = m->scratch;
  float* svec = m->scratch + (size_t)B * m->hd.D;
  return run_modulation(m, t, B, table, (hipStream_t)stream, hid, svec);
}

int sf_residual(sf_model* m, const float* x, const float* t, int B, const sf_cond* cond, int blocks, float* hout,
                void* stream) {
  if (!m) return SF_E_NOTLOADED;
  if (!x || !t || !hout || B < 1 || B > SF_MAX_ROWS || !finite_all(t, B) || blocks < 0 ||
      blocks > (int)m->hd.L)
    return SF_E_INVAL;
  bool guided;
  float w;
  const int rows = rows_for(m, B, cond, &guided, &w);
  if (!rows) return SF_E_INVAL;
  hipStream_t s = (hipStream_t)stream;
  SF_TRY(note_modulation(m, t, B, s, run_network(m, x, t, B, rows, cond, blocks, nullptr, s)));
  if (hipMemcpyAsync(hout, m->h, sizeof(float) * (size_t)rows * m->N * m->hd.D, hipMemcpyDeviceToDevice, s) !=
      hipSuccess)
    return SF_E_HIP;
  return SF_OK;
}

int sf_attention(sf_model* m, const void* q, const void* k, const void* vT, void* o, int rows, void* stream) {
  if (!m) return SF_E_NOTLOADED;
  if (!q || !k || !vT || !o || rows < 1 || rows > SF_MAX_ROWS) return SF_E_INVAL;
  const Header& h = m->hd;
  sf::AttnArgs a{q, k, vT, o, rows, (int)h.heads, m->N, m->N, m->dh, m->ldv, (int)h.D,
                 (float)(1.0 / std::sqrt((double)m->dh)), m->vperm};
  return sf::launch_attention(m->bf16, a, (hipStream_t)stream) == hipSuccess ? SF_OK : SF_E_HIP;
}

int sf_debug_read(sf_model* m, int buffer, void* dst, size_t bytes, void* stream) {
  if (!m) return SF_E_NOTLOADED;
  if (!dst) return SF_E_INVAL;
  const Header& h = m->hd;
  const size_t R = m->max_rows, D = h.D, M = R * m->N;
  const void* src = nullptr;
  size_t cap = 0;
  switch (buffer) {
    case SF_BUF_H: src = m->h; cap = M * D * 4; break;
    case SF_BUF_ACT: src = m->act; cap = M * D * m->es; break;
    case SF_BUF_Q: src = m->q; cap = M * D * m->es; break;
    case SF_BUF_K: src = m->k; cap = M * D * m->es; break;
    case SF_BUF_VT: src = m->vT; cap = R * D * m->ldv * m->es; break;
    case SF_BUF_ATTN: src = m->o; cap = M * D * m->es; break;
    case SF_BUF_MLP: src = m->f; cap = M * h.mlp * m->es; break;
    case SF_BUF_TABLE: src = m->table; cap = R * m->modw * 4; break;
    default: return SF_E_INVAL;
  }
  if (bytes > cap) return SF_E_INVAL;
  if (hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, (hipStream_t)stream) != hipSuccess) return SF_E_HIP;
  return SF_OK;
}

int sf_timing_enable(sf_model* m, int kc, int enable) {
  if (!m) return SF_E_NOTLOADED;
  if (kc < 0 || kc >= SF_KC_COUNT) return SF_E_INVAL;
  Timing& tm = m->timing[kc];
  if (enable && tm.ev.empty()) {
    tm.ev.resize(2 * kTimingPool);
    for (auto& e : tm.ev)
      if (hipEventCreate(&e) != hipSuccess) return SF_E_HIP;
  }
  tm.on = enable != 0;
  tm.used = 0;
  tm.launches = 0;
  return SF_OK;
}

int sf_timing_read(sf_model* m, int kc, double* total_ms, long* launches) {
  if (!m) return SF_E_NOTLOADED;
  if (kc < 0 || kc >= SF_KC_COUNT || !total_ms || !launches) return SF_E_INVAL;
  Timing& tm = m->timing[kc];
  double sum = 0.0;
  for (int i = 0; i < tm.used; ++i) {
    if (hipEventSynchronize(tm.ev[2 * i + 1]) != hipSuccess) return SF_E_HIP;
    float ms = 0.0f;
    if (hipEventElapsedTime(&ms, tm.ev[2 * i], tm.ev[2 * i + 1]) != hipSuccess) return SF_E_HIP;
    sum += ms;
  }
  *total_ms = sum;
  *launches = tm.used;
  tm.used = 0;
  tm.launches = 0;
  return SF_OK;
}

int sf_graph_enable(sf_model* m, int enable) {
  if (!m) return SF_E_NOTLOADED;
  if (!enable && !m->graphs.empty()) {
    if (hipDeviceSynchronize() != hipSuccess) return SF_E_HIP;
    drop_graphs(m);
  }
  m->graph_on = enable != 0;
  return SF_OK;
}

int sf_modulation_cache(sf_model* m, int enable) {
  if (!m) return SF_E_NOTLOADED;
  m->mod_cache_on = enable != 0;
  m->mod_valid = false;
  return SF_OK;
}

int sf_context_cache(sf_model* m, int enable) {
  if (!m) return SF_E_NOTLOADED;
  if (m->ctx_st) {
    if (hipDeviceSynchronize() != hipSuccess || sf::launch_ctx_reset(m->ctx_st, nullptr) != hipSuccess ||
        hipDeviceSynchronize() != hipSuccess)
      return SF_E_HIP;
  }
  m->ctx_cache_on = enable != 0;
  return SF_OK;
}

int sf_context_cache_stats(const sf_model* m, long* calls, long* computed) {
  if (!m) return SF_E_NOTLOADED;
  if (!calls || !computed) return SF_E_INVAL;
  *calls = 0;
  *computed = 0;
  if (!m->ctx_st) return SF_OK;
  sf::CtxState st;
  if (hipDeviceSynchronize() != hipSuccess || hipMemcpy(&st, m->ctx_st, sizeof(st), hipMemcpyDeviceToHost) != hipSuccess)
    return SF_E_HIP;
  *calls = (long)st.calls;
  *computed = (long)st.computed;
  return SF_OK;
}

int sf_modulation_cache_stats(const sf_model* m, long* skips) {
  if (!m) return SF_E_NOTLOADED;
  if (!skips) return SF_E_INVAL;
  *skips = m->mod_skips;
  return SF_OK;
}

int sf_graph_stats(const sf_model* m, int* cached, long* replays) {
  if (!m) return SF_E_NOTLOADED;
  if (!cached || !replays) return SF_E_INVAL;
  *cached = (int)m->graphs.size();
  *replays = m->graph_replays;
  return SF_OK;
}

int sf_set_scheduler(sf_model* m, const sf_perflow* p) {
  if (!m) return SF_E_NOTLOADED;
  if (!p) {
    if (m->windows != 0 && !m->graphs.empty()) {
      if (hipDeviceSynchronize() != hipSuccess) return SF_E_HIP;
      drop_graphs(m);
    }
    m->windows = 0;
    return SF_OK;
  }
  if (p->windows < 1 || p->windows > 4096 || p->train_steps < 2 || p->train_steps > (1 << 20) ||
      !(p->beta_start > 0.0f) || !(p->beta_end > p->beta_start) || !(p->beta_end < 1.0f) ||
      !(p->eps >= 0.0) || !(p->eps < 1.0 / p->windows))
    return SF_E_INVAL;
  // scaled-linear schedule: sqrt(beta) on a linear grid (start + i * step, the last
  // point exactly the end), beta = its square, alphas_cumprod = running product of 1 - beta
  const int T = p->train_steps;
  const double s0 = std::sqrt((double)p->beta_start), s1 = std::sqrt((double)p->beta_end);
  const double step = (s1 - s0) / (double)(T - 1);
  std::vector<double> ab((size_t)T);
  double prod = 1.0;
  for (int i = 0; i < T; ++i) {
    const double sb = i == T - 1 ? s1 : (double)i * step + s0;
    prod *= 1.0 - sb * sb;
    ab[(size_t)i] = prod;
  }
  if (hipDeviceSynchronize() != hipSuccess) return SF_E_HIP;
  drop_graphs(m);
  // the scheduler is off until the new schedule is in place: a failure below leaves
  // Euler on the velocity, never a window count without its schedule
  m->windows = 0;
  if (m->n_abar != T) {
    if (m->abar) (void)hipFree(m->abar);
    m->abar = nullptr;
    m->n_abar = 0;
    if (fail_alloc_after() == 0 || hipMalloc((void**)&m->abar, sizeof(double) * (size_t)T) != hipSuccess) {
      m->abar = nullptr;
      (void)hipGetLastError();
      return SF_E_OOM;
    }
    m->n_abar = T;
  }
  if (hipMemcpy(m->abar, ab.data(), sizeof(double) * (size_t)T, hipMemcpyHostToDevice) != hipSuccess)
    return SF_E_HIP;
  m->win_eps = p->eps;
  m->windows = p->windows;
  return SF_OK;
}

int sf_scheduler_shift(sf_model* m, float* x, const float* out, const float* t, const float* dt, int B,
                       const float* z_new, float* x_done, void* stream) {
  if (!m) return SF_E_NOTLOADED;
  if (!x || !out || !t || !dt || !z_new || B < 1 || B > SF_MAX_ROWS || !finite_all(t, B) || !finite_all(dt, B))
    return SF_E_INVAL;
  hipStream_t s = (hipStream_t)stream;
  return timed(m, SF_KC_EULER, s, [&]() {
    sf::EulerArgs a{};
    a.x = x; a.v = out; a.B = B; a.E = m->E; a.guided = 0; a.w = 0.0f;
    for (int i = 0; i < B; ++i) a.dt.v[i] = dt[i];
    a.z_new = z_new; a.x_done = x_done;
    set_windows(m, t, B, a);
    return sf::launch_euler_shift(a, s);
  });
}

int sf_noise_latent(sf_model* m, const float* x_ref, const float* z, float t0, float* out, void* stream) {
  if (!m) return SF_E_NOTLOADED;
  if (!x_ref || !z || !out || !(t0 >= 0.0f && t0 <= 1.0f)) return SF_E_INVAL;
  return sf::launch_noise_latent(x_ref, z, t0, m->E, out, (hipStream_t)stream) == hipSuccess ? SF_OK : SF_E_HIP;
}

}  // extern "C"
