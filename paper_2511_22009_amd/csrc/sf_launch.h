// Internal interface between the C-ABI runtime (streamflow.cpp) and the gfx950
// kernels: argument structs and launchers. Not part of the public ABI.
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sf {

// Events that the next kernel launched from this host thread attaches to its own
// dispatch packet, so they hold that kernel's start and end timestamps rather than
// those of the stream around it. launch() consumes them (one kernel only).
struct LaunchEvents {
  hipEvent_t start;
  hipEvent_t stop;
};
extern thread_local LaunchEvents t_launch_events;

template <typename F, typename... Args>
inline void launch(F kernel, dim3 grid, dim3 block, uint32_t lds, hipStream_t s, Args... args) {
  const LaunchEvents ev = t_launch_events;
  t_launch_events = LaunchEvents{nullptr, nullptr};
  hipExtLaunchKernelGGL(kernel, grid, block, lds, s, ev.start, ev.stop, 0u, args...);
}

constexpr int kMaxRows = 64;     // equals SF_MAX_ROWS
constexpr int kOffOOBHost = 0x7ffffff0;  // the device code's past-the-end buffer offset
constexpr int kMaxWidth = 2048;  // largest D / mlp input width a row kernel holds
constexpr int kMaxPatch = 32;    // largest p*p*C

// Per-row scalars passed by value in the kernel argument block (t or dt of each slot).
struct RowScalars {
  float v[kMaxRows];
};

// Division by a divisor fixed for a launch: q = (umulhi(n, magic) + n) >> shift,
// exact for every 32-bit n (magic from the round-up method for invariant divisors).
struct FastDiv {
  uint32_t magic;
  uint32_t shift;
  uint32_t d;
};
FastDiv make_fastdiv(uint32_t d);

// ---- K1: batched GEMV  Y[b][j] = act(W[j,:] . X[b,:] + bias[j]) ------------------
// x_mode 1 builds X on the fly as the sinusoidal embedding of 1000 t[b] (width K,
// [cos | sin] over K/2 frequencies `freqs`).
struct GemvArgs {
  const void* W;        // [R][K], bf16 or fp32
  const float* bias;    // [R]
  const float* X;       // [B][ldx] (x_mode 0)
  int ldx;
  int B, K, R;
  float* Y;             // [B][ldy]
  int ldy;
  int act;              // 0 identity, 1 SiLU
  int x_mode;           // 0 memory, 1 sinusoid of 1000 t
  const float* freqs;   // [K/2] (x_mode 1)
  RowScalars t;         // (x_mode 1)
};
hipError_t launch_gemv(bool w_bf16, const GemvArgs& a, hipStream_t s);
// Device address (on the current device) and size in floats of the fixed scratch array
// of the allocation-free conditioning call; looked up once per device.
hipError_t modulation_scratch(float** out, size_t* floats);

// ---- K2: patchify + patch embed + position table ---------------------------------
struct EmbedArgs {
  const float* x;       // [n_lat][C][H][W]
  int n_lat;            // network row r reads latent r % n_lat
  const float* W_pe;    // [P][D] (transposed patch-embedding weight)
  const float* b_pe;    // [D]
  const float* pos;     // [N][D]
  float* h;             // [rows*N][D]
  int rows, C, H, W, p, D, N;
};
hipError_t launch_embed(const EmbedArgs& a, hipStream_t s);
// The last adaLN projection (x_mode 0) and the patch embed in one launch, each part with
// the arithmetic of its own kernel. Supported for 2x2 patches of 4 channels and GEMV
// rows of at most three chunks per lane; otherwise hipErrorInvalidValue, nothing launched.
bool gemv_embed_supported(bool w_bf16, const GemvArgs& g, const EmbedArgs& e);
hipError_t launch_gemv_embed(bool w_bf16, const GemvArgs& g, const EmbedArgs& e, hipStream_t s);

// ---- context entries of the cross-attention K/V ------------------------------------
// The keys and values of a context depend on the context and the weights only, so they
// are computed per ENTRY (one context) for every block at once, and each network row
// reads the entry of its context through kv_map: the B conditional rows their own
// contexts, every unconditional row the one null-context entry. Device-side state of
// the entries (one block of ints in the workspace):
struct CtxState {
  int kv_map[kMaxRows];        // network row -> entry
  int prev_slot[kMaxRows];     // entry of each conditional slot in the previous call
  int flags[kMaxRows + 1];     // per context row of a call: bit 0 / bit 1 set when it
                               // differs from the entry of the same / the previous slot
  int live[kMaxRows + 1];      // entries whose keys and values this call computes
  int src[kMaxRows + 1];       // the context row that fills a live entry
  int prev_B;                  // conditional slots of the previous call (0: none known)
  int prev_null;               // entry of the null context in the previous call + 1
  unsigned long long calls;    // calls through the entry lookup
  unsigned long long computed; // entries computed by them
};
struct CtxArgs {
  const float* ctx;       // [B][ctx_len][ctx_dim]
  const float* null_ctx;  // [ctx_len][ctx_dim] (guided) or nullptr
  int B, guided;          // context rows of the call: B, plus one null row if guided
  int per_row;            // ctx_len * ctx_dim
  int n_entries;          // entries held (max_rows + 1)
  float* keep;            // [n_entries][per_row]: the context each entry was computed from
  void* ctxA;             // [n_entries][pitch]: the same in the compute type (GEMM operand);
  int pitch;              // pitch = ctx_len rounded up to 16 tokens, x ctx_dim (zero rows)
  CtxState* st;
};
// Without reuse: entries 0..B-1 take the conditional contexts, entry B the null
// context; kv_map accordingly. One kernel.
hipError_t launch_ctx_prepare(bool use_bf16, const CtxArgs& a, hipStream_t s);
// With reuse: each context row is compared bitwise with the entry its slot held in the
// previous call and with the entry of the previous slot (where Alg. 2's shift moved it);
// a row equal to either reuses that entry, the others take entries no row of this call
// uses, which are marked live and filled. Three kernels (compare, assign, fill).
hipError_t launch_ctx_lookup(bool use_bf16, const CtxArgs& a, hipStream_t s);
// Forgets every entry (no row of the next call can reuse one).
hipError_t launch_ctx_reset(CtxState* st, hipStream_t s);

// ---- K5: LayerNorm (+ per-sample adaLN modulate) ---------------------------------
struct LnArgs {
  const float* h;       // [M][D] fp32 residual stream
  void* out;            // [M][D] bf16 or fp32
  int M, D;
  const float* table;   // adaLN table [n_slots][ldt], or nullptr for plain LN
  int ldt, shift_off, scale_off;
  FastDiv tok;          // divides a token row index by N -> network row
  int n_slots;          // network row r uses table row (r < n_slots ? r : r - n_slots)
};
hipError_t launch_ln(bool out_bf16, const LnArgs& a, hipStream_t s);

// ---- K7: final LN + modulate + linear D -> p*p*C + unpatchify ----------------------
struct HeadArgs {
  const float* h;       // [rows*N][D]
  const float* W_f;     // [P][D]
  const float* b_f;     // [P]
  const float* table;
  int ldt, shift_off, scale_off;
  int n_slots;
  FastDiv tok;
  float* v;             // [rows][C][H][W]
  int rows, C, H, W, p, D, N, P;
};
hipError_t launch_head(const HeadArgs& a, hipStream_t s);

// ---- K3: GEMM  C[M][N] = A[M][K] . B[N][K]^T with a fused epilogue -----------------
enum EpiKind {
  EPI_QKV = 0,       // + bias, scatter to head-major q / k and transposed v
  EPI_RES_GATE = 1,  // h += gate[slot][n] * (acc + bias)
  EPI_GELU = 2,      // out = GELU_tanh(acc + bias)
  EPI_RES = 3,       // h += acc + bias
  EPI_RES_GATE_MLP = 4, // EPI_RES_GATE for the MLP down-projection (a separate kernel
                        // symbol, so profiles tell it from the attention projection)
  EPI_KVX = 5           // + bias, the context keys / transposed values of every block:
                        // column n is block (n / D) / 2, key if (n / D) even else value
};
struct GemmArgs {
  const void* A;
  int lda;
  const void* B;
  int ldb;
  int M, N, K;
  const float* bias;
  // EPI_QKV: column n of the projection is part (which_base + n / D) of {q, k, v},
  // head (n % D) / dh, dim (n % D) % dh; row m is token m % ntok of network row m / ntok.
  void* q;
  void* k;
  void* vT;             // [rows][heads][dh][ldv]; token t at column t, or at vt_pos(t) if vperm
  int heads, dh, D, ntok, ldv, which_base, vperm;
  FastDiv div_ntok, div_D, div_dh;
  // EPI_KVX: number of blocks L; the keys of block b for network row r land at row
  // r * L + b of q/k's [rows][heads][ntok][dh] layout (likewise vT)
  int kv_blocks;
  // optional (EPI_KVX): a tile whose rows m all have row_live[m / ntok] == 0 is skipped
  const int* row_live;
  // EPI_RES_GATE / EPI_RES
  float* h;
  int ldh;
  const float* table;
  int ldt, gate_off, n_slots;
  // EPI_GELU
  void* out;
  int ldo;
};
hipError_t launch_gemm(bool use_bf16, EpiKind kind, const GemmArgs& a, hipStream_t s);
// The same with an explicit bf16 tile shape (index into the tile table; -1 = choose).
hipError_t launch_gemm_tile(bool use_bf16, int tile, EpiKind kind, const GemmArgs& a, hipStream_t s);
int choose_gemm_tile(int M, int N, int K);

// ---- K4: softmax attention per (network row, head) ---------------------------------
// Column of key t in the permuted transposed-v layout: bits 2 and 3 of t swapped, so in
// every group of 16 keys the columns hold keys 0-3, 8-11, 4-7, 12-15. Eight adjacent
// columns then hold the eight keys one lane half feeds into a 16-key step of the P.V
// product (keys 4g..4g+3 and 8+4g..8+4g+3 for lane half g), read as one 16-byte
// fragment. An involution; needs ldv to be a multiple of 16.
__host__ __device__ constexpr int vt_pos(int t) { return (t & ~12) | ((t & 4) << 1) | ((t & 8) >> 1); }

struct AttnArgs {
  const void* q;        // [rows][heads][Nq][dh]
  const void* k;        // [rows][heads][Nk][dh]
  const void* vT;       // [rows][heads][dh][ldv], columns of no key are zero; key t at
                        // column t, or at vt_pos(t) if vperm (the bf16 kernels)
  void* o;              // [rows][Nq][D], head j at columns j*dh ..
  int rows, heads, Nq, Nk, dh, ldv, D;
  float scale;          // 1 / sqrt(dh)
  int vperm;
  // optional: row r reads the keys and values of row kv_map[r] (nullptr: row r), whose
  // k starts k_rs elements after the previous row's and vT v_rs after (0: heads*k_ld*dh
  // and heads*dh*ldv, the packed layout); k holds k_ld >= Nk key rows per head (0: Nk),
  // the rows past Nk unread
  const int* kv_map;
  size_t k_rs, v_rs;
  int k_ld;
};
hipError_t launch_attention(bool use_bf16, const AttnArgs& a, hipStream_t s);
bool attention_supports(int dh);

// ---- K6: guidance combine + Euler update + queue shift -----------------------------
struct EulerArgs {
  float* x;             // [B(+1)][E] slots, updated in place
  const float* v;       // [B][E], or [2B][E] (cond rows then uncond rows) with guidance
  int B, E;
  int guided;
  float w;
  RowScalars dt;
  const float* z_new;   // [E]
  float* x_done;        // [E] or nullptr (filling: the queue grows to B+1)
  // windows > 0: v is a noise prediction and the update is the time-window conversion
  // (x' = x + dt (lambda_t x + eta_t v - x) / (t^e - t)), per slot from t, the window
  // count, the lookup tolerance and alphas_cumprod [n_abar] (fp64)
  int windows;
  double eps;
  const double* abar;
  int n_abar;
  RowScalars t;
};
hipError_t launch_euler_shift(const EulerArgs& a, hipStream_t s);
// v_out[k] = v[B+k] + w (v[k] - v[B+k]) for k < B.
hipError_t launch_cfg_combine(const float* v, int B, int E, float w, float* v_out, hipStream_t s);
// out = (1 - t0) x_ref + t0 z, each product and the sum rounded separately
hipError_t launch_noise_latent(const float* x_ref, const float* z, float t0, int E, float* out, hipStream_t s);

}  // namespace sf
