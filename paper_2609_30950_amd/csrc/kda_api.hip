// C ABI of libkda: argument validation, workspace layout and launches.
// Declarations and argument contracts: include/kda.h.

#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <cstring>

#include "../../include/kda.h"
#include "kda_kernels.hpp"
#include "kda_profile.hpp"

namespace {

using kda::KParams;

struct WsLayout {
  size_t c_off, zr_off, bits_off, s32_off, rpart_off, gam_off, hv_off, chunk_off, total;
};

size_t up256(size_t x) { return (x + 255) / 256 * 256; }

WsLayout ws_layout(const kda_config* cfg) {
  const size_t rows = (size_t)cfg->B * cfg->H * cfg->d_k;
  WsLayout w;
  w.c_off = 0;
  w.zr_off = up256(w.c_off + rows * sizeof(double));
  w.bits_off = up256(w.zr_off + rows * sizeof(uint32_t));
  w.s32_off = up256(w.bits_off + rows);
  // prefill: per-slice row maxima (d_v / 64 slices) and the rows' weights Gamma
  w.rpart_off = up256(w.s32_off + rows * (size_t)cfg->d_v * sizeof(float));
  w.gam_off = up256(w.rpart_off + rows * (size_t)(cfg->d_v / 64) * sizeof(float));
  // decode: the token's vectors w (d_v), a and g (d_k) per head
  w.hv_off = up256(w.gam_off + rows * sizeof(double));
  w.chunk_off = up256(w.hv_off + (size_t)cfg->B * cfg->H * (cfg->d_v + 2 * cfg->d_k) * sizeof(float));
  // chunked prefill: the records of two groups of chunks (the next group is
  // prepared while the current one is applied)
  const int nbh = cfg->B * cfg->H;
  const size_t chunk =
      cfg->chunked ? (size_t)2 * kda::chunk_group(nbh) * nbh * kda::chunk_record_bytes(cfg->d_k) : 0;
  w.total = up256(w.chunk_off + chunk);
  return w;
}

// Validate a config; fills the budget of one scope unit.
int check_cfg(const kda_config* cfg, int* need) {
  if (cfg == nullptr) return KDA_ERR_ARG;
  if (cfg->B < 1 || cfg->H < 1) return KDA_ERR_SHAPE;
  if (cfg->d_k != cfg->d_v) return KDA_ERR_UNSUPPORTED;
  if (cfg->d_k != 64 && cfg->d_k != 128 && cfg->d_k != 256) return KDA_ERR_UNSUPPORTED;
  if (cfg->decay_per_head != 0 && cfg->decay_per_head != 1) return KDA_ERR_ARG;
  if (cfg->state32 != 0 && cfg->state32 != 1) return KDA_ERR_ARG;
  if (cfg->no_erase != 0 && cfg->no_erase != 1) return KDA_ERR_ARG;
  if (cfg->chunked != 0 && cfg->chunked != 1) return KDA_ERR_ARG;
  if (cfg->chunked && (cfg->d_k > 128 || cfg->state32)) return KDA_ERR_UNSUPPORTED;
  if (cfg->head_units != 0 && cfg->head_units != 1) return KDA_ERR_ARG;
  if (cfg->weight_mode < KDA_WEIGHT_EMA || cfg->weight_mode > KDA_WEIGHT_DECAY) return KDA_ERR_ARG;
  // head widths come from the statistics alone (R~ = 1): no range variants
  if (cfg->head_units && (cfg->weight_mode == KDA_WEIGHT_RANGE ||
                          cfg->weight_mode == KDA_WEIGHT_GAMMA_RANGE ||
                          cfg->weight_mode == KDA_WEIGHT_REL_RANGE))
    return KDA_ERR_UNSUPPORTED;
  if (cfg->head_units) {
    // one width per head, block scales: per-head normalisation, the layer
    // budget over the heads of a sequence, widths 2..8
    if (cfg->state32 || cfg->chunked) return KDA_ERR_UNSUPPORTED;
    if (cfg->group_rows != cfg->d_k || cfg->scope != KDA_SCOPE_SEQUENCE) return KDA_ERR_ARG;
    if (cfg->b_min < 2 || cfg->b_max < cfg->b_min || cfg->b_max > 8) return KDA_ERR_ARG;
    if (cfg->ema_span < 1 || !std::isfinite(cfg->mean_bits)) return KDA_ERR_ARG;
    if (cfg->H > 4096) return KDA_ERR_UNSUPPORTED;
    const long long K = (long long)std::floor(cfg->mean_bits * (double)cfg->H + 0.5);
    if (K < (long long)cfg->H * cfg->b_min || K > (long long)cfg->H * cfg->b_max) return KDA_ERR_ARG;
    if (need) *need = (int)(K - (long long)cfg->H * cfg->b_min);
    return KDA_OK;
  }
  if (cfg->state32) {
    if (need) *need = 0;
    return KDA_OK;
  }
  if (cfg->scope != KDA_SCOPE_SEQUENCE && cfg->scope != KDA_SCOPE_HEAD) return KDA_ERR_ARG;
  if (cfg->group_rows < 1) return KDA_ERR_ARG;
  if (cfg->group_rows <= cfg->d_k) {
    if (cfg->d_k % cfg->group_rows != 0) return KDA_ERR_ARG;
  } else {
    // groups spanning heads: whole heads, inside one sequence's budget
    if (cfg->group_rows % cfg->d_k != 0 || (cfg->H * cfg->d_k) % cfg->group_rows != 0 ||
        cfg->scope != KDA_SCOPE_SEQUENCE)
      return KDA_ERR_ARG;
  }
  if (cfg->b_min < 1 || cfg->b_max < cfg->b_min || cfg->b_max > 16) return KDA_ERR_ARG;
  if (cfg->d_k == 256 && cfg->b_max > 8) return KDA_ERR_UNSUPPORTED;   // LDS code tile
  if (cfg->ema_span < 1) return KDA_ERR_ARG;
  if (!std::isfinite(cfg->mean_bits)) return KDA_ERR_ARG;
  const long long N = cfg->scope == KDA_SCOPE_SEQUENCE ? (long long)cfg->H * cfg->d_k : cfg->d_k;
  if (N > 4096) return KDA_ERR_UNSUPPORTED;
  const long long K = (long long)std::floor(cfg->mean_bits * (double)N + 0.5);
  if (K < N * cfg->b_min || K > N * cfg->b_max) return KDA_ERR_ARG;
  if (need) *need = (int)(K - N * cfg->b_min);
  return KDA_OK;
}

KParams make_params(const kda_config* cfg, int need) {
  KParams p;
  std::memset(&p, 0, sizeof(p));
  p.B = cfg->B;
  p.H = cfg->H;
  p.dk = cfg->d_k;
  p.dv = cfg->d_v;
  p.G = cfg->group_rows;
  p.scope = cfg->scope;
  p.bmin = cfg->b_min;
  p.bmax = cfg->b_max;
  p.per_head = cfg->decay_per_head;
  p.state32 = cfg->state32;
  p.no_erase = cfg->no_erase;
  p.weight_mode = cfg->weight_mode;
  p.wb_C = 1;
  p.need = need;
  p.alpha = 2.0 / (double)(cfg->ema_span + 1);
  p.one_minus_alpha = 1.0 - p.alpha;
  p.L = cfg->head_units ? kda::make_head_layout(cfg->d_k, cfg->d_v, cfg->b_max)
                        : kda::make_layout(cfg->d_k, cfg->d_v, cfg->b_max < 1 ? 1 : cfg->b_max);
  p.diag_fit = kda::prof_counter();
  for (int b = 0; b <= kda::MAX_B; ++b)
    for (int m = 0; m < kda::N_FIT; ++m) {
      const int n = b >= 2 ? (1 << (b - 1)) - 1 : 0;
      p.phi[b][m] = n > 0 ? (float)((double)(5 + m) / (double)(20 * n)) : 0.f;
    }
  return p;
}

void set_ws(KParams& p, const kda_config* cfg, void* ws) {
  const WsLayout w = ws_layout(cfg);
  uint8_t* base = (uint8_t*)ws;
  p.ws_c = (double*)(base + w.c_off);
  p.ws_zr = (uint32_t*)(base + w.zr_off);
  p.ws_bits = base + w.bits_off;
  p.ws_s32 = (float*)(base + w.s32_off);
  p.ws_rpart = (float*)(base + w.rpart_off);
  p.ws_gam = (double*)(base + w.gam_off);
  p.ws_hv = (float*)(base + w.hv_off);
  p.ws_chunk = cfg->chunked ? base + w.chunk_off : nullptr;
}

int hip_status(hipError_t e) { return e == hipSuccess ? KDA_OK : KDA_ERR_HIP; }

// ------------------------------------------------ allocation-free step ---
// Scratch of kda_step_noalloc: a file-scope device array (one copy per GPU
// the library runs on, held until the process ends).  Host code never uses
// the array's name as a device address; it uses the address that
// hipGetSymbolAddress returns for the current device, kept per device.
constexpr size_t KDA_SCRATCH_BYTES = (size_t)16 << 20;
__device__ __align__(256) unsigned char scratch[KDA_SCRATCH_BYTES];
constexpr int SCRATCH_MAX_DEV = 64;
std::atomic<void*> g_scratch_addr[SCRATCH_MAX_DEV];

// Device address of this device's scratch (nullptr on a HIP error).  Calls
// that race here compute the same address.
void* scratch_address() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= SCRATCH_MAX_DEV) return nullptr;
  void* ptr = g_scratch_addr[dev].load(std::memory_order_acquire);
  if (ptr == nullptr) {
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    g_scratch_addr[dev].store(ptr, std::memory_order_release);
  }
  return ptr;
}

// Views of the decode step (d_k <= 128, per-row units) inside the scratch:
// keys, rate codes, widths, per-slice row maxima, Gamma and the token's
// vectors; no float32 state (the requantisation rebuilds it).
WsLayout scratch_layout(const kda_config* cfg) {
  const size_t rows = (size_t)cfg->B * cfg->H * cfg->d_k;
  WsLayout w;
  w.c_off = 0;
  w.zr_off = up256(w.c_off + rows * sizeof(double));
  w.bits_off = up256(w.zr_off + rows * sizeof(uint32_t));
  w.s32_off = up256(w.bits_off + rows);
  w.rpart_off = w.s32_off;
  w.gam_off = up256(w.rpart_off + rows * (size_t)(cfg->d_v / 64) * sizeof(float));
  w.hv_off = up256(w.gam_off + rows * sizeof(double));
  w.chunk_off = up256(w.hv_off + (size_t)cfg->B * cfg->H * (cfg->d_v + 2 * cfg->d_k) * sizeof(float));
  w.total = w.chunk_off;
  return w;
}

// Kernels use 16-byte vector accesses on records, workspace and states.
bool aligned16(const void* ptr) { return ((uintptr_t)ptr & 15u) == 0; }

}  // namespace

extern "C" {

size_t kda_record_bytes(const kda_config* cfg) {
  if (check_cfg(cfg, nullptr) != KDA_OK) return 0;
  if (cfg->state32) return (size_t)cfg->d_k * cfg->d_v * sizeof(float);
  if (cfg->head_units) return (size_t)kda::make_head_layout(cfg->d_k, cfg->d_v, cfg->b_max).slot;
  return (size_t)kda::make_layout(cfg->d_k, cfg->d_v, cfg->b_max).slot;
}

size_t kda_workspace_bytes(const kda_config* cfg) {
  if (check_cfg(cfg, nullptr) != KDA_OK) return 0;
  return ws_layout(cfg).total;
}

const char* kda_status_str(int status) {
  switch (status) {
    case KDA_OK: return "ok";
    case KDA_ERR_ARG: return "invalid argument";
    case KDA_ERR_SHAPE: return "invalid shape";
    case KDA_ERR_UNSUPPORTED: return "unsupported configuration";
    case KDA_ERR_WORKSPACE: return "workspace missing";
    case KDA_ERR_HIP: return "HIP launch or runtime error";
    default: return "unknown status";
  }
}

int kda_weights(const kda_config* cfg, int32_t W, int32_t C, const float* q, const float* s,
                const float* beta, const float* k, double* gamma, void* stream) {
  int need = 0;
  int st = check_cfg(cfg, &need);
  if (st != KDA_OK) return st;
  if (W < 1 || C < 1) return KDA_ERR_ARG;
  if (!q || !s || !beta || !k || !gamma) return KDA_ERR_ARG;
  KParams p = make_params(cfg, need);
  return hip_status(kda::launch_window_gamma(p, W, C, q, s, beta, k, gamma, (hipStream_t)stream));
}

int kda_weights_exact(const kda_config* cfg, int32_t W, int32_t C, const float* q, const float* s,
                      const float* beta, const float* k, double* gamma, void* stream) {
  int need = 0;
  int st = check_cfg(cfg, &need);
  if (st != KDA_OK) return st;
  if (W < 1 || C < 1) return KDA_ERR_ARG;
  if (!q || !s || !beta || !k || !gamma) return KDA_ERR_ARG;
  if (cfg->d_k > 128) return KDA_ERR_UNSUPPORTED;   // the float64 matrix per head
  KParams p = make_params(cfg, need);
  return hip_status(kda::launch_exact_gamma(p, W, C, q, s, beta, k, gamma, (hipStream_t)stream));
}

int kda_alloc_bits(const kda_config* cfg, const double* gamma, const float* R, uint8_t* bits,
                   void* ws, void* stream) {
  int need = 0;
  int st = check_cfg(cfg, &need);
  if (st != KDA_OK) return st;
  if (cfg->state32) return KDA_ERR_ARG;
  if (cfg->head_units) return KDA_ERR_UNSUPPORTED;
  if (!gamma || !R || !bits) return KDA_ERR_ARG;
  if (!ws) return KDA_ERR_WORKSPACE;
  KParams p = make_params(cfg, need);
  set_ws(p, cfg, ws);
  return hip_status(kda::launch_alloc_bits(p, gamma, R, bits, (hipStream_t)stream));
}

int kda_pack_state(const kda_config* cfg, const float* S, const uint8_t* bits, const double* s_hat,
                   const double* r, uint32_t tokens_seen, void* records, void* stream) {
  int need = 0;
  int st = check_cfg(cfg, &need);
  if (st != KDA_OK) return st;
  if (cfg->state32) return KDA_ERR_ARG;
  if (cfg->head_units) return KDA_ERR_UNSUPPORTED;
  if (!S || !bits || !s_hat || !r || !records) return KDA_ERR_ARG;
  if (!aligned16(S) || !aligned16(records)) return KDA_ERR_ARG;
  KParams p = make_params(cfg, need);
  p.records = records;
  return hip_status(kda::launch_pack(p, S, bits, s_hat, r, tokens_seen, (hipStream_t)stream));
}

int kda_unpack_state(const kda_config* cfg, const void* records, float* S, uint8_t* bits,
                     double* s_hat, double* r, void* stream) {
  int need = 0;
  int st = check_cfg(cfg, &need);
  if (st != KDA_OK) return st;
  if (!records || !aligned16(records)) return KDA_ERR_ARG;
  if (cfg->head_units) return KDA_ERR_UNSUPPORTED;
  if (cfg->state32 && (bits || s_hat || r)) return KDA_ERR_ARG;
  KParams p = make_params(cfg, need);
  p.records = const_cast<void*>(records);
  return hip_status(kda::launch_unpack(p, S, bits, s_hat, r, (hipStream_t)stream));
}

// Checked parameters of a decode step (phase: 1 outputs, 2 write-back, 3 both).
static int step_params(const kda_config* cfg, void* records, const float* q, const float* k,
                       const float* v, const float* s, const float* beta, const double* gamma,
                       float* o, void* ws, int phase, KParams* out) {
  int need = 0;
  int st = check_cfg(cfg, &need);
  if (st != KDA_OK) return st;
  if (!records) return KDA_ERR_ARG;
  if ((phase & 1) && (!q || !k || !v || !s || !beta || !o)) return KDA_ERR_ARG;
  if (!cfg->state32 && !ws) return KDA_ERR_WORKSPACE;
  if (!aligned16(records) || (ws && !aligned16(ws))) return KDA_ERR_ARG;
  KParams p = make_params(cfg, need);
  p.records = records;
  p.q = q;
  p.k = k;
  p.v = v;
  p.s = s;
  p.beta = beta;
  p.gamma = gamma;
  p.o = o;
  p.T = 1;
  p.tok0 = 0;
  p.ntk = 1;
  p.in_bf16 = 0;
  if (!cfg->state32) set_ws(p, cfg, ws);
  *out = p;
  return KDA_OK;
}

int kda_step(const kda_config* cfg, void* records, const float* q, const float* k, const float* v,
             const float* s, const float* beta, const double* gamma, float* o, void* ws,
             void* stream) {
  KParams p;
  const int st = step_params(cfg, records, q, k, v, s, beta, gamma, o, ws, 3, &p);
  if (st != KDA_OK) return st;
  if (cfg->head_units) return hip_status(kda::launch_step_heads(p, (hipStream_t)stream));
  return hip_status(kda::launch_step(p, (hipStream_t)stream));
}

int kda_step_noalloc(const kda_config* cfg, void* records, const float* q, const float* k,
                     const float* v, const float* s, const float* beta, const double* gamma,
                     float* o, void* stream) {
  int need = 0;
  const int st = check_cfg(cfg, &need);
  if (st != KDA_OK) return st;
  if (cfg->state32)   // the unquantised step needs no scratch
    return kda_step(cfg, records, q, k, v, s, beta, gamma, o, nullptr, stream);
  if (cfg->head_units || cfg->d_k > 128) return KDA_ERR_UNSUPPORTED;
  if (scratch_layout(cfg).total > KDA_SCRATCH_BYTES) return KDA_ERR_WORKSPACE;
  void* ws = scratch_address();
  if (ws == nullptr) return KDA_ERR_HIP;
  KParams p;
  const int ps = step_params(cfg, records, q, k, v, s, beta, gamma, o, ws, 3, &p);
  if (ps != KDA_OK) return ps;
  const WsLayout w = scratch_layout(cfg);
  uint8_t* base = (uint8_t*)ws;
  p.ws_c = (double*)(base + w.c_off);
  p.ws_zr = (uint32_t*)(base + w.zr_off);
  p.ws_bits = base + w.bits_off;
  p.ws_s32 = nullptr;
  p.ws_rpart = (float*)(base + w.rpart_off);
  p.ws_gam = (double*)(base + w.gam_off);
  p.ws_hv = (float*)(base + w.hv_off);
  p.ws_chunk = nullptr;
  return hip_status(kda::launch_step(p, (hipStream_t)stream));
}

size_t kda_step_noalloc_max_bytes(void) { return KDA_SCRATCH_BYTES; }

int kda_step_outputs(const kda_config* cfg, void* records, const float* q, const float* k,
                     const float* v, const float* s, const float* beta, const double* gamma,
                     float* o, void* ws, void* stream) {
  KParams p;
  const int st = step_params(cfg, records, q, k, v, s, beta, gamma, o, ws, 1, &p);
  if (st != KDA_OK) return st;
  if (cfg->head_units) return KDA_ERR_UNSUPPORTED;
  return hip_status(kda::launch_step_outputs(p, (hipStream_t)stream));
}

int kda_step_writeback(const kda_config* cfg, void* records, void* ws, void* stream) {
  KParams p;
  const int st = step_params(cfg, records, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                             nullptr, ws, 2, &p);
  if (st != KDA_OK) return st;
  if (cfg->head_units) return KDA_ERR_UNSUPPORTED;
  return hip_status(kda::launch_step_writeback(p, (hipStream_t)stream));
}

int kda_gate_quant(const kda_config* cfg, int32_t T, int32_t bits, int32_t mode, const float* s,
                   float* s_out, void* stream) {
  if (cfg == nullptr) return KDA_ERR_ARG;
  if (cfg->B < 1 || cfg->H < 1) return KDA_ERR_SHAPE;
  if (T < 1) return KDA_ERR_ARG;
  if (cfg->d_k != 64 && cfg->d_k != 128 && cfg->d_k != 256) return KDA_ERR_UNSUPPORTED;
  if (cfg->decay_per_head) return KDA_ERR_UNSUPPORTED;
  if (bits < 1 || bits > 16 || (mode != KDA_GATES_LOG && mode != KDA_GATES_LINEAR)) return KDA_ERR_ARG;
  if (!s || !s_out) return KDA_ERR_ARG;
  KParams p;
  std::memset(&p, 0, sizeof(p));
  p.B = cfg->B;
  p.H = cfg->H;
  p.dk = cfg->d_k;
  return hip_status(kda::launch_gate_quant(p, T, bits, mode == KDA_GATES_LINEAR, s, s_out,
                                           (hipStream_t)stream));
}

int kda_prefill_aux(const kda_config* cfg, int32_t T, int32_t C, void* records, const uint16_t* q,
                    const uint16_t* k, const uint16_t* v, const float* s, const float* beta,
                    const double* gamma, float* o, void* ws, void* stream, void* aux_stream) {
  int need = 0;
  int st = check_cfg(cfg, &need);
  if (st != KDA_OK) return st;
  if (T < 1 || C < 1) return KDA_ERR_ARG;
  if (!records || !q || !k || !v || !s || !beta || !o) return KDA_ERR_ARG;
  if (!cfg->state32 && !ws) return KDA_ERR_WORKSPACE;
  if (!aligned16(records) || (ws && !aligned16(ws))) return KDA_ERR_ARG;
  KParams p = make_params(cfg, need);
  p.records = records;
  p.q = q;
  p.k = k;
  p.v = v;
  p.s = s;
  p.beta = beta;
  p.gamma = gamma;
  p.o = o;
  p.T = T;
  p.in_bf16 = 1;
  p.wb_C = C;
  if (!cfg->state32) set_ws(p, cfg, ws);
  if (cfg->chunked) {
    if (C > 64) return KDA_ERR_ARG;
    return hip_status(kda::launch_prefill_chunked(p, C, (hipStream_t)stream, (hipStream_t)aux_stream));
  }
  if (cfg->head_units) return hip_status(kda::launch_prefill_heads(p, C, (hipStream_t)stream));
  return hip_status(kda::launch_prefill(p, C, (hipStream_t)stream));
}

int kda_prefill(const kda_config* cfg, int32_t T, int32_t C, void* records, const uint16_t* q,
                const uint16_t* k, const uint16_t* v, const float* s, const float* beta,
                const double* gamma, float* o, void* ws, void* stream) {
  return kda_prefill_aux(cfg, T, C, records, q, k, v, s, beta, gamma, o, ws, stream, nullptr);
}

}  // extern "C"
