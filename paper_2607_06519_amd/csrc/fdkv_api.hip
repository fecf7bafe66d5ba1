// C ABI of libfdkv: host-side validation, the closed-form cache layout, the
// routing rule of Eq. (3) with the budget search of Section 3, and the
// launches of the HIP kernels on the caller's stream.
#include <math.h>
#include <stdio.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <vector>

#include "fdkv.h"
#include "fdkv_common.h"
#include "fdkv_kernels.h"

using namespace fdkv;

namespace {

thread_local std::string g_last_error;

bool aligned(const void* p, uintptr_t a) { return p && ((reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0); }

// bytes per input / exact-plane element, and per stored coefficient
int elem_bytes(const fdkv_dims* d) { return d->dtype == FDKV_F32 ? 4 : 2; }
int coef_bytes(const fdkv_dims* d) { return d->dtype == FDKV_F32 ? 4 : d->dtype == FDKV_BF16 ? 2 : 1; }

// Blocks of a schedule: first layer and size of each, in layer order.
struct Sched {
  int n;
  int first[kMaxBlocks], size[kMaxBlocks];
};

// Section 4: blocks of four by default, pairs for the first and the last
// four layers (MIXED); all pairs or all fours otherwise.
bool make_sched(int L, int schedule, Sched* out) {
  Sched s{};
  auto add = [&](int B) {
    s.first[s.n] = s.n ? s.first[s.n - 1] + s.size[s.n - 1] : 0;
    s.size[s.n++] = B;
  };
  if (schedule == FDKV_SCHED_PAIRS) {
    if (L < 2 || L % 2) return false;
    for (int i = 0; i < L / 2; ++i) add(2);
  } else if (schedule == FDKV_SCHED_QUADS) {
    if (L < 4 || L % 4) return false;
    for (int i = 0; i < L / 4; ++i) add(4);
  } else if (schedule == FDKV_SCHED_MIXED) {
    if (L < 8 || (L - 8) % 4) return false;
    add(2);
    add(2);
    for (int i = 0; i < (L - 8) / 4; ++i) add(4);
    add(2);
    add(2);
  } else {
    return false;
  }
  *out = s;
  return true;
}

// The blocks of one size, as a kernel block list.
BlockList blocks_of_size(const Sched& s, int B) {
  BlockList bl{};
  for (int i = 0; i < s.n; ++i)
    if (s.size[i] == B) {
      bl.block[bl.n] = (int16_t)i;
      bl.first[bl.n] = (int16_t)s.first[i];
      ++bl.n;
    }
  return bl;
}

// Weight of a stored residual value of frequency j = 1..3 at position p of
// a block: B = 2 stores the layer-0 image D of the half difference (+1 at
// p = 0, -1 at p = 1); B = 4 stores the coefficient Z_j, weighted by
// F_4[j][p] = cos(pi (2p + 1) j / 8) / sqrt(2).
void layer_weights(int B, int p, float w[3]) {
  for (int j = 1; j <= 3; ++j)
    w[j - 1] = B == 2 ? (p ? -1.f : 1.f) : (float)(cos(M_PI * (2 * p + 1) * j / 8.0) / sqrt(2.0));
}

fdkv_status check_dims(const fdkv_dims* d) {
  if (!d) return FDKV_E_INVALID_ARG;
  if (d->n_layers < 2 || d->n_layers > kMaxPtrLayers) return FDKV_E_INVALID_ARG;
  Sched sch;
  if (!make_sched(d->n_layers, d->schedule, &sch)) return FDKV_E_INVALID_ARG;
  if (d->n_kv_heads < 1 || d->n_q_heads < d->n_kv_heads || d->n_q_heads % d->n_kv_heads) return FDKV_E_INVALID_ARG;
  if (d->head_dim < 1 || d->head_dim > 256) return FDKV_E_INVALID_ARG;
  if (d->topk < 0 || d->topk > d->head_dim) return FDKV_E_INVALID_ARG;
  if (d->dtype != FDKV_F32 && d->dtype != FDKV_BF16 && d->dtype != FDKV_BF16_E4M3) return FDKV_E_INVALID_ARG;
  if (d->residual != FDKV_RES_CHANNELS && d->residual != FDKV_RES_TOKENS) return FDKV_E_INVALID_ARG;
  if (d->residual == FDKV_RES_TOKENS && (d->res_ppm < 0 || d->res_ppm > 1000000)) return FDKV_E_INVALID_ARG;
  if (d->n_rates < 0 || d->n_rates > kMaxRates || (d->n_rates > 0 && d->residual != FDKV_RES_TOKENS))
    return FDKV_E_INVALID_ARG;
  for (int j = 0; j < d->n_rates; ++j)
    if (d->rates_ppm[j] < 0 || d->rates_ppm[j] > 1000000 || (j > 0 && d->rates_ppm[j] <= d->rates_ppm[j - 1]))
      return FDKV_E_INVALID_ARG;
  if (d->head_dim != 64 && d->head_dim != 128) return FDKV_E_UNSUPPORTED;
  const int G = d->n_q_heads / d->n_kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8) return FDKV_E_UNSUPPORTED;
  return FDKV_OK;
}

fdkv_status hip_fail(hipError_t e, const char* what) {
  g_last_error = std::string(what) + ": " + hipGetErrorString(e);
  return FDKV_E_HIP;
}

uint64_t bytes_per_token(int mode, int d, int k, int e, int c, int B) {
  if (mode == kShared) return 2ull * d * c;
  if (mode == kResidual) return 2ull * d * c + 2ull * k * (index_bytes(B) + c);
  return 2ull * B * d * e;
}

bool tokens_mode(const fdkv_dims* d) { return d->residual == FDKV_RES_TOKENS; }

// The fraction of tokens of a residual unit's set, from its mode byte.
int ppm_of(const fdkv_dims* dm, uint32_t byte) { return unit_ppm(dm->res_ppm, dm->n_rates, dm->rates_ppm, byte); }

// Average bytes per token of a mode for Omega: the token-level residual pays
// r of the (B - 1) high-frequency rows of K and V plus its 1-bit mask and a
// uint32 count per 128 tokens.
double omega_bytes(const fdkv_dims* dm, int mode, int B, int ppm) {
  const int d = dm->head_dim, e = elem_bytes(dm), c = coef_bytes(dm);
  if (tokens_mode(dm) && mode == kResidual)
    return 2.0 * d * c + 2.0 * (B - 1) * d * c * (ppm / 1e6) + 1.0 / 8 + 4.0 / kTokChunk;
  return (double)bytes_per_token(mode, d, dm->topk, e, c, B);
}

// Bytes of a segment of the unit with mode byte `byte`.
uint64_t segment_bytes(const fdkv_dims* dm, uint32_t byte, uint64_t T, int B) {
  const int e = elem_bytes(dm), c = coef_bytes(dm);
  if (tokens_mode(dm)) return tok_layout(mode_of(byte), T, dm->head_dim, ppm_of(dm, byte), e, c, B).total;
  return seg_layout(mode_of(byte), T, dm->head_dim, dm->topk, e, c, B).total;
}

// Largest fraction a set of this cache can keep.
int max_ppm(const fdkv_dims* dm) { return dm->n_rates ? dm->rates_ppm[dm->n_rates - 1] : dm->res_ppm; }

Sched sched_of(const fdkv_dims* d) {
  Sched s{};
  make_sched(d->n_layers, d->schedule, &s);
  return s;
}

uint64_t probe_chunks(int T) { return (uint64_t)(T + kProbeChunk - 1) / kProbeChunk; }

// Probe workspace: probe Gram matrices per (layer, KV head) and per-chunk
// partials (every block finds its top-k inside its Gram kernel).
struct ProbeWs {
  uint64_t gram, part, total;
};
ProbeWs probe_ws_layout(const fdkv_dims* d, int T) {
  const Sched sch = sched_of(d);
  const uint64_t units = (uint64_t)sch.n * d->n_kv_heads;
  ProbeWs w{};
  if (tokens_mode(d)) {  // the token scores' sums of squares
    w.total = plane_bytes(units * (uint64_t)T * 4);
    return w;
  }
  w.gram = 0;
  w.part = w.gram + plane_bytes((uint64_t)d->n_layers * d->n_kv_heads * d->head_dim * d->head_dim * 4);
  w.total = w.part + plane_bytes(units * probe_chunks(T) * 2 * 4);
  return w;
}

uint64_t decode_chunks(int max_T) { return (uint64_t)(max_T + kDecodeWgTokens - 1) / kDecodeWgTokens; }

// The split-K records of fdkv_decode_attn_static live in this file-scope
// device array, one copy per GPU, held until the process ends.  Host code
// never passes the array's name to a kernel (on the host it is only a
// stand-in for the symbol): each device's address comes from
// hipGetSymbolAddress, taken once per device with that device current.
constexpr size_t kStaticScratchBytes = size_t(16) << 20;
constexpr int kMaxDevices = 64;
__device__ __align__(256) uint8_t scratch[kStaticScratchBytes];
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

fdkv_status scratch_of_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    g_last_error = std::string("hipGetDevice: ") + hipGetErrorString(e);
    return FDKV_E_HIP;
  }
  if (dev < 0 || dev >= kMaxDevices) {
    g_last_error = "fdkv_decode_attn_static: device index beyond the static scratch table";
    return FDKV_E_UNSUPPORTED;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      g_last_error = std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e);
      return FDKV_E_HIP;
    }
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return FDKV_OK;
}

}  // namespace

extern "C" {

const char* fdkv_status_string(int32_t s) {
  switch (s) {
    case FDKV_OK: return "ok";
    case FDKV_E_INVALID_ARG: return "invalid argument";
    case FDKV_E_UNSUPPORTED: return "unsupported shape (head_dim must be 64 or 128, Hq/Hkv in 1,2,4,8)";
    case FDKV_E_WORKSPACE: return "workspace too small";
    case FDKV_E_BUDGET: return "byte budget below the all-shared footprint";
    case FDKV_E_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char* fdkv_last_error(void) { return g_last_error.c_str(); }

fdkv_status fdkv_blocks(const fdkv_dims* dims, int32_t* n_blocks, int32_t* first_layer, int32_t* block_size) {
  fdkv_status st = check_dims(dims);
  if (st != FDKV_OK) return st;
  if (!n_blocks) return FDKV_E_INVALID_ARG;
  const Sched s = sched_of(dims);
  *n_blocks = s.n;
  for (int i = 0; i < s.n; ++i) {
    if (first_layer) first_layer[i] = s.first[i];
    if (block_size) block_size[i] = s.size[i];
  }
  return FDKV_OK;
}

fdkv_status fdkv_layout(const fdkv_dims* dims, int32_t batch, const int32_t* seq_lens, const uint8_t* modes,
                        uint64_t* seg_offsets, uint64_t* total_bytes) {
  fdkv_status st = check_dims(dims);
  if (st != FDKV_OK) return st;
  if (batch < 1 || !seq_lens || !modes || !total_bytes) return FDKV_E_INVALID_ARG;
  const Sched sch = sched_of(dims);
  const int units = sch.n * dims->n_kv_heads;
  for (int b = 0; b < batch; ++b) {
    if (seq_lens[b] < 0) return FDKV_E_INVALID_ARG;
    for (int u = 0; u < units; ++u)
      if (!unit_byte_ok(modes[(size_t)b * units + u], tokens_mode(dims) ? dims->n_rates : 0)) return FDKV_E_INVALID_ARG;
  }
  const int e = elem_bytes(dims), c = coef_bytes(dims);
  uint64_t off = 0;
  for (int b = 0; b < batch; ++b)
    for (int u = 0; u < units; ++u) {
      const size_t i = (size_t)b * units + u;
      if (seg_offsets) seg_offsets[i] = off;
      off += segment_bytes(dims, modes[i], (uint64_t)seq_lens[b], sch.size[u / dims->n_kv_heads]);
    }
  *total_bytes = off;
  return FDKV_OK;
}

#pragma clang fp contract(off)
fdkv_status fdkv_route(const fdkv_dims* dims, int32_t seq_len, const float* errors, double lambda,
                       uint64_t budget_bytes, uint8_t* modes_out, double* lambda_out) {
  fdkv_status st = check_dims(dims);
  if (st != FDKV_OK) return st;
  if (seq_len < 0 || !errors || !modes_out) return FDKV_E_INVALID_ARG;
  if (budget_bytes == 0 && !(lambda >= 0.0)) return FDKV_E_INVALID_ARG;
  const Sched sch = sched_of(dims);
  const int units = sch.n * dims->n_kv_heads;
  // Candidates of a unit: shared, the residual mode (at every routed fraction,
  // or at its one fraction), exact.  Per block size: Omega, segment bytes,
  // mode byte and the column of the errors array that holds the loss (-1: 0).
  const int J = tokens_mode(dims) && dims->n_rates ? dims->n_rates : 1;
  const int C = J + 2, stride = 1 + J;
  double om[2][kMaxRates + 2];
  uint64_t seg[2][kMaxRates + 2];
  uint8_t byte[kMaxRates + 2];
  int col[kMaxRates + 2];
  for (int c = 0; c < C; ++c) {
    byte[c] = (uint8_t)(c == 0 ? kShared : c == C - 1 ? kExact : (kResidual | ((J > 1 || dims->n_rates ? c - 1 : 0) << 2)));
    col[c] = c == C - 1 ? -1 : c;
  }
  for (int bi = 0; bi < 2; ++bi) {
    const int B = bi ? 4 : 2;
    const double full = omega_bytes(dims, kExact, B, 0);
    for (int c = 0; c < C; ++c) {
      om[bi][c] = omega_bytes(dims, mode_of(byte[c]), B, ppm_of(dims, byte[c])) / full;
      seg[bi][c] = segment_bytes(dims, byte[c], (uint64_t)seq_len, B);
    }
  }
  auto quad = [&](int u) { return sch.size[u / dims->n_kv_heads] == 4 ? 1 : 0; };
  auto loss = [&](int u, int c) { return col[c] < 0 ? 0.0 : (double)errors[(size_t)u * stride + col[c]]; };
  // Of two candidates, the cheaper one first (equal cost: the lower candidate).
  auto order = [](const double* o, int m1, int m2, int& a, int& b) {
    const bool first = o[m1] < o[m2] || (o[m1] == o[m2] && m1 < m2);
    a = first ? m1 : m2;
    b = first ? m2 : m1;
  };

  // argmin of E_c + lambda Omega_c, ties to the cheaper candidate.  Two
  // candidates are compared through their breakpoint (E_a - E_b) / (Omega_b -
  // Omega_a): the cheaper wins iff lambda >= it.  At a candidate lambda equal
  // to a unit's breakpoint its two candidates tie exactly (the same expression
  // gives both numbers), where the two costs evaluated in floating point might
  // round apart.
  auto decide = [&](double lam, uint8_t* out) {
    uint64_t fp = 0;
    for (int u = 0; u < units; ++u) {
      const double* o = om[quad(u)];
      int best = 0;
      for (int c = 1; c < C; ++c) {
        int a, b;
        order(o, best, c, a, b);
        const double Ea = loss(u, a), Eb = loss(u, b);
        const bool cheaper_wins = o[a] == o[b] ? Ea <= Eb : lam >= (Ea - Eb) / (o[b] - o[a]);
        best = cheaper_wins ? a : b;
      }
      out[u] = byte[best];
      fp += seg[quad(u)][best];
    }
    return fp;
  };

  if (budget_bytes == 0) {
    decide(lambda, modes_out);
    if (lambda_out) *lambda_out = lambda;
    return FDKV_OK;
  }
  std::vector<double> cands;
  cands.push_back(0.0);
  for (int u = 0; u < units; ++u) {
    const double* o = om[quad(u)];
    for (int i = 0; i < C; ++i)
      for (int j = i + 1; j < C; ++j) {
        int a, b;
        order(o, i, j, a, b);
        if (!(o[b] > o[a])) continue;
        const double lam = (loss(u, a) - loss(u, b)) / (o[b] - o[a]);
        if (lam > 0.0 && isfinite(lam)) cands.push_back(lam);
      }
  }
  std::sort(cands.begin(), cands.end());
  cands.erase(std::unique(cands.begin(), cands.end()), cands.end());
  cands.push_back(INFINITY);
  std::vector<uint8_t> tmp((size_t)units);
  for (double lam : cands) {
    if (decide(lam, tmp.data()) <= budget_bytes) {
      std::copy(tmp.begin(), tmp.end(), modes_out);
      if (lambda_out) *lambda_out = lam;
      return FDKV_OK;
    }
  }
  std::fill(modes_out, modes_out + units, (uint8_t)FDKV_SHARED);
  if (lambda_out) *lambda_out = INFINITY;
  return FDKV_E_BUDGET;
}
#pragma clang fp contract(on)

fdkv_status fdkv_probe_workspace(const fdkv_dims* dims, int32_t seq_len, int32_t n_probe, size_t* bytes) {
  fdkv_status st = check_dims(dims);
  if (st != FDKV_OK) return st;
  if (seq_len < 1 || n_probe < 1 || !bytes) return FDKV_E_INVALID_ARG;
  *bytes = (size_t)probe_ws_layout(dims, seq_len).total;
  return FDKV_OK;
}

// Bytes per input piece of the probe's K selections: a 32-bit mask when the
// schedule has blocks of four (3 CPP coefficients a piece), else a byte.
int selection_slot_bytes(const Sched& sch) {
  for (int i = 0; i < sch.n; ++i)
    if (sch.size[i] == 4) return 4;
  return 1;
}

fdkv_status fdkv_selection_bytes(const fdkv_dims* dims, int32_t seq_len, size_t* bytes) {
  fdkv_status st = check_dims(dims);
  if (st != FDKV_OK) return st;
  if (seq_len < 0 || !bytes) return FDKV_E_INVALID_ARG;
  const Sched sch = sched_of(dims);
  *bytes = (size_t)((uint64_t)sch.n * dims->n_kv_heads * (uint64_t)seq_len *
                    selection_pieces(dims->head_dim, elem_bytes(dims)) * selection_slot_bytes(sch));
  return FDKV_OK;
}

fdkv_status fdkv_probe(const fdkv_dims* dims, int32_t seq_len, const void* const* k_layers,
                       const void* const* qp_layers, int32_t n_probe, float* errors_out, float* token_scores_out,
                       void* ws, size_t ws_bytes, uint8_t* k_select_out, void* stream) {
  fdkv_status st = check_dims(dims);
  if (st != FDKV_OK) return st;
  if (seq_len < 1 || n_probe < 1 || !k_layers || !qp_layers) return FDKV_E_INVALID_ARG;
  // key planes and each head's probe rows are addressed with 32-bit offsets
  const uint64_t row_bytes = (uint64_t)dims->head_dim * elem_bytes(dims);
  if ((uint64_t)seq_len * row_bytes >= (1ull << 31) ||
      (uint64_t)n_probe * (dims->n_q_heads / dims->n_kv_heads) * row_bytes >= (1ull << 31))
    return FDKV_E_UNSUPPORTED;
  if (!aligned(errors_out, 4) || !aligned(ws, 256) || (k_select_out && !aligned(k_select_out, 4)))
    return FDKV_E_INVALID_ARG;
  for (int l = 0; l < dims->n_layers; ++l)
    if (!aligned(k_layers[l], 16) || !aligned(qp_layers[l], 16)) return FDKV_E_INVALID_ARG;
  const ProbeWs w = probe_ws_layout(dims, seq_len);
  if (ws_bytes < w.total) return FDKV_E_WORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  uint8_t* base = static_cast<uint8_t*>(ws);

  const Sched sch = sched_of(dims);
  if (tokens_mode(dims)) {
    if (!aligned(token_scores_out, 4)) return FDKV_E_INVALID_ARG;
    TokenParams tp{};
    for (int l = 0; l < dims->n_layers; ++l) {
      tp.k[l] = k_layers[l];
      tp.qp[l] = qp_layers[l];
    }
    tp.modes = nullptr;
    tp.scores = token_scores_out;
    tp.sumsq = reinterpret_cast<float*>(base);
    tp.errors = errors_out;
    tp.seq_len = seq_len;
    tp.hkv = dims->n_kv_heads;
    tp.hq = dims->n_q_heads;
    tp.d = dims->head_dim;
    tp.n_probe = n_probe;
    tp.res_ppm = dims->res_ppm;
    tp.n_rates = dims->n_rates;
    for (int j = 0; j < dims->n_rates; ++j) tp.rates_ppm[j] = dims->rates_ppm[j];
    tp.bf16 = dims->dtype != FDKV_F32;
    for (int B = 2; B <= 4; B += 2) {
      tp.bl = blocks_of_size(sch, B);
      tp.bsize = B;
      if (tp.bl.n == 0) continue;
      hipError_t e = launch_token_scores(tp, s);
      if (e != hipSuccess) return hip_fail(e, "token_scores");
      e = launch_token_select(tp, s);
      if (e != hipSuccess) return hip_fail(e, "token_select");
    }
    return FDKV_OK;
  }
  ProbeParams pp{};
  for (int l = 0; l < dims->n_layers; ++l) {
    pp.k[l] = k_layers[l];
    pp.qp[l] = qp_layers[l];
  }
  pp.ksel = k_select_out;
  pp.ksel_bytes = selection_slot_bytes(sch);
  pp.gram_q = reinterpret_cast<float*>(base + w.gram);
  pp.partial = reinterpret_cast<float*>(base + w.part);
  pp.errors = errors_out;
  pp.seq_len = seq_len;
  pp.n_blocks = sch.n;
  for (int i = 0; i < sch.n; ++i) pp.bsizes[i] = (int8_t)sch.size[i];
  pp.hkv = dims->n_kv_heads;
  pp.hq = dims->n_q_heads;
  pp.d = dims->head_dim;
  pp.topk = dims->topk;
  pp.n_probe = n_probe;
  pp.n_chunks = (int)probe_chunks(seq_len);
  pp.bf16 = dims->dtype != FDKV_F32;
  for (int B = 2; B <= 4; B += 2) {
    pp.bl = blocks_of_size(sch, B);
    pp.bsize = B;
    if (pp.bl.n == 0) continue;
    const hipError_t e = launch_probe(pp, s);  // every block takes its top-k inside its Gram kernel
    if (e != hipSuccess) return hip_fail(e, "probe");
  }
  const hipError_t e = launch_probe_finalize(pp, s);
  if (e != hipSuccess) return hip_fail(e, "probe_finalize");
  return FDKV_OK;
}

fdkv_status fdkv_compress(const fdkv_dims* dims, int32_t seq_len, const void* const* k_layers,
                          const void* const* v_layers, const uint8_t* modes, const uint64_t* seg_offsets,
                          const float* token_scores, const uint8_t* k_select, void* cache, void* stream) {
  fdkv_status st = check_dims(dims);
  if (st != FDKV_OK) return st;
  if (seq_len < 0 || !k_layers || !v_layers || !modes || !aligned(seg_offsets, 8) || !aligned(cache, 256))
    return FDKV_E_INVALID_ARG;
  for (int l = 0; l < dims->n_layers; ++l)
    if (!aligned(k_layers[l], 16) || !aligned(v_layers[l], 16)) return FDKV_E_INVALID_ARG;
  if (seq_len == 0) return FDKV_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);

  const Sched sch = sched_of(dims);
  CompressParams cp{};
  for (int l = 0; l < dims->n_layers; ++l) {
    cp.k[l] = k_layers[l];
    cp.v[l] = v_layers[l];
  }
  cp.modes = modes;
  cp.seg_off = seg_offsets;
  cp.cache = static_cast<uint8_t*>(cache);
  cp.seq_len = seq_len;
  cp.hkv = dims->n_kv_heads;
  cp.d = dims->head_dim;
  cp.topk = dims->topk;
  cp.bf16 = dims->dtype != FDKV_F32;
  cp.coef8 = dims->dtype == FDKV_BF16_E4M3;
  const bool tok = tokens_mode(dims);
  cp.tokres = tok;
  cp.ksel = tok ? nullptr : k_select;
  cp.ksel_bytes = selection_slot_bytes(sch);
  if (tok && !aligned(token_scores, 4)) return FDKV_E_INVALID_ARG;
  if (!tok && k_select && !aligned(k_select, 4)) return FDKV_E_INVALID_ARG;
  TokenParams tp{};
  for (int l = 0; l < dims->n_layers; ++l) {
    tp.k[l] = k_layers[l];
    tp.v[l] = v_layers[l];
  }
  tp.modes = modes;
  tp.seg_off = seg_offsets;
  tp.cache = cp.cache;
  tp.scores = const_cast<float*>(token_scores);
  tp.seq_len = seq_len;
  tp.hkv = cp.hkv;
  tp.hq = dims->n_q_heads;
  tp.d = cp.d;
  tp.res_ppm = dims->res_ppm;
  tp.n_rates = dims->n_rates;
  for (int j = 0; j < dims->n_rates; ++j) tp.rates_ppm[j] = dims->rates_ppm[j];
  tp.bf16 = cp.bf16;
  tp.coef8 = cp.coef8;
  for (int B = 2; B <= 4; B += 2) {
    cp.bl = tp.bl = blocks_of_size(sch, B);
    cp.bsize = tp.bsize = B;
    if (cp.bl.n == 0) continue;
    hipError_t e = launch_compress_dense(cp, s);
    if (e != hipSuccess) return hip_fail(e, "compress_dense");
    if (tok) {
      e = launch_token_select(tp, s);
      if (e != hipSuccess) return hip_fail(e, "token_select");
      e = launch_token_rows(tp, s);
      if (e != hipSuccess) return hip_fail(e, "token_rows");
    }  // per-token channel residuals: the dense pass takes their entries
  }
  return FDKV_OK;
}

fdkv_status fdkv_decode_workspace(const fdkv_dims* dims, int32_t batch, int32_t max_seq_len, size_t* bytes) {
  return fdkv_decode_spans_workspace(dims, batch, 1, &max_seq_len, -1, bytes);
}

fdkv_status fdkv_decode_spans_workspace(const fdkv_dims* dims, int32_t batch, int32_t n_spans,
                                        const int32_t* max_seq_lens, int32_t tail_cap, size_t* bytes) {
  fdkv_status st = check_dims(dims);
  if (st != FDKV_OK) return st;
  if (batch < 1 || n_spans < 0 || n_spans + (tail_cap >= 0 ? 1 : 0) > kMaxParts || !bytes ||
      (n_spans > 0 && !max_seq_lens))
    return FDKV_E_INVALID_ARG;
  uint64_t n = 0;
  for (int i = 0; i < n_spans; ++i) {
    if (max_seq_lens[i] < 0) return FDKV_E_INVALID_ARG;
    n += decode_chunks(max_seq_lens[i]);
  }
  if (tail_cap >= 0) n += decode_chunks(tail_cap);
  const uint64_t G = dims->n_q_heads / dims->n_kv_heads;
  *bytes = (size_t)((uint64_t)batch * dims->n_kv_heads * std::max<uint64_t>(n, 1) * G * (dims->head_dim + 4) * 4);
  return FDKV_OK;
}

fdkv_status fdkv_append(const fdkv_dims* dims, int32_t batch, const int32_t* pos, int32_t cap, const void* k_new,
                        const void* v_new, void* tail_k, void* tail_v, void* stream) {
  fdkv_status st = check_dims(dims);
  if (st != FDKV_OK) return st;
  if (batch < 1 || cap < 1 || !aligned(pos, 4) || !aligned(k_new, 16) || !aligned(v_new, 16) ||
      !aligned(tail_k, 16) || !aligned(tail_v, 16))
    return FDKV_E_INVALID_ARG;
  AppendParams ap{};
  ap.pos = pos;
  ap.k_new = k_new;
  ap.v_new = v_new;
  ap.tail_k = tail_k;
  ap.tail_v = tail_v;
  ap.batch = batch;
  ap.hkv = dims->n_kv_heads;
  ap.cap = cap;
  ap.row_bytes = dims->head_dim * elem_bytes(dims);
  const hipError_t e = launch_append(ap, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "append");
  return FDKV_OK;
}

fdkv_status fdkv_check_conversions(uint64_t* mismatches, void* stream) {
  if (!mismatches) return FDKV_E_INVALID_ARG;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  unsigned long long* counts = nullptr;
  hipError_t e = hipMalloc(&counts, 2 * sizeof(unsigned long long));
  if (e != hipSuccess) return hip_fail(e, "check_conversions");
  unsigned long long host[2] = {0ull, 0ull};
  e = hipMemsetAsync(counts, 0, sizeof(host), s);
  if (e == hipSuccess) e = launch_check_conversions(counts, s);
  if (e == hipSuccess) e = hipMemcpyAsync(host, counts, sizeof(host), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  const hipError_t ef = hipFree(counts);
  if (e == hipSuccess) e = ef;
  if (e != hipSuccess) return hip_fail(e, "check_conversions");
  mismatches[0] = host[0];
  mismatches[1] = host[1];
  return FDKV_OK;
}

}  // extern "C"

namespace {

// Decode phases: the split-K pass that writes the records, the merge of the records into the outputs.
enum : int { kPhaseSplit = 1, kPhaseMerge = 2 };

fdkv_status decode_impl(const fdkv_dims* dims, int32_t batch, int32_t n_spans, const fdkv_span* spans,
                        const fdkv_tail* tail, int32_t layer, const void* q, void* out, float sm_scale, void* ws,
                        size_t ws_bytes, void* stream, int phases) {
  fdkv_status st = check_dims(dims);
  if (st != FDKV_OK) return st;
  const int n_parts = n_spans + (tail ? 1 : 0);
  if (batch < 1 || n_spans < 0 || n_parts > kMaxParts || (n_spans > 0 && !spans) || layer < 0 ||
      layer >= dims->n_layers)
    return FDKV_E_INVALID_ARG;
  if (!aligned(q, 16) || ((phases & kPhaseMerge) && !aligned(out, 16)) || !aligned(ws, 16) || !isfinite(sm_scale))
    return FDKV_E_INVALID_ARG;
  const uint64_t row = (uint64_t)dims->head_dim * elem_bytes(dims);
  int32_t maxes[kMaxParts];
  for (int i = 0; i < n_spans; ++i) {
    const fdkv_span& sp = spans[i];
    if (sp.max_seq_len < 0 || !aligned(sp.seq_lens, 4) || !aligned(sp.modes, 4) || !aligned(sp.seg_offsets, 8) ||
        !aligned(sp.cache, 256))
      return FDKV_E_INVALID_ARG;
    if ((uint64_t)sp.max_seq_len * row >= (1ull << 31)) return FDKV_E_UNSUPPORTED;
    // the rows of a token-level residual set are addressed with 32-bit offsets too
    if (tokens_mode(dims) && residual_token_count((uint64_t)sp.max_seq_len, max_ppm(dims)) * 3 * row >= (1ull << 31))
      return FDKV_E_UNSUPPORTED;
    maxes[i] = sp.max_seq_len;
  }
  if (tail) {
    if (tail->cap < 0 || !aligned(tail->lens, 4) || !aligned(tail->k, 16) || !aligned(tail->v, 16))
      return FDKV_E_INVALID_ARG;
    if ((uint64_t)tail->cap * row >= (1ull << 31)) return FDKV_E_UNSUPPORTED;
  }
  size_t need = 0;
  st = fdkv_decode_spans_workspace(dims, batch, n_spans, maxes, tail ? tail->cap : -1, &need);
  if (st != FDKV_OK) return st;
  if (ws_bytes < need) return FDKV_E_WORKSPACE;

  DecodeParams p{};
  p.q = q;
  p.out = out;
  p.ws = static_cast<float*>(ws);
  const Sched sch = sched_of(dims);
  int blk = 0;
  while (!(layer < sch.first[blk] + sch.size[blk])) ++blk;
  p.block = blk;
  p.pos = layer - sch.first[blk];
  p.bsize = sch.size[blk];
  layer_weights(p.bsize, p.pos, p.wres);
  p.n_blocks = sch.n;
  p.hkv = dims->n_kv_heads;
  p.hq = dims->n_q_heads;
  p.d = dims->head_dim;
  p.topk = dims->topk;
  p.batch = batch;
  p.scale_log2 = sm_scale * 1.4426950408889634f;
  p.bf16 = dims->dtype != FDKV_F32;
  p.coef8 = dims->dtype == FDKV_BF16_E4M3;
  p.tokres = tokens_mode(dims);
  p.res_ppm = dims->res_ppm;
  p.n_rates = dims->n_rates;
  for (int j = 0; j < dims->n_rates; ++j) p.rates_ppm[j] = dims->rates_ppm[j];
  // record slots: every part's chunks, spans first, then the tail
  int total = 0;
  for (int i = 0; i < n_parts; ++i) {
    const bool t = i == n_spans;
    p.part[i].base = total;
    p.part[i].chunks = (int)decode_chunks(t ? tail->cap : spans[i].max_seq_len);
    p.part[i].lens = t ? tail->lens : spans[i].seq_lens;
    if (!t) {
      p.part[i].cache = static_cast<const uint8_t*>(spans[i].cache);
      p.part[i].modes = spans[i].modes;
      p.part[i].seg_off = spans[i].seg_offsets;
    }
    total += p.part[i].chunks;
  }
  p.n_parts = n_parts;
  p.n_chunks_total = total;
  p.tail_part = tail ? n_spans : -1;
  if (tail) {
    p.tail_k = tail->k;
    p.tail_v = tail->v;
    p.tail_cap = tail->cap;
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (total > 0 && (phases & kPhaseSplit)) {
    const hipError_t e = launch_decode(p, s);
    if (e != hipSuccess) return hip_fail(e, "decode");
  }
  if (phases & kPhaseMerge) {
    const hipError_t e = launch_decode_merge(p, s);
    if (e != hipSuccess) return hip_fail(e, "decode_merge");
  }
  return FDKV_OK;
}

}  // namespace

extern "C" {

fdkv_status fdkv_decode_spans(const fdkv_dims* dims, int32_t batch, int32_t n_spans, const fdkv_span* spans,
                              const fdkv_tail* tail, int32_t layer, const void* q, void* out, float sm_scale,
                              void* ws, size_t ws_bytes, void* stream) {
  return decode_impl(dims, batch, n_spans, spans, tail, layer, q, out, sm_scale, ws, ws_bytes, stream,
                     kPhaseSplit | kPhaseMerge);
}

fdkv_status fdkv_decode_partial(const fdkv_dims* dims, int32_t batch, const int32_t* seq_lens, int32_t max_seq_len,
                                const uint8_t* modes, const uint64_t* seg_offsets, const void* cache, int32_t layer,
                                const void* q, float sm_scale, void* ws, size_t ws_bytes, void* stream) {
  fdkv_status st = check_dims(dims);
  if (st != FDKV_OK) return st;
  if (max_seq_len < 0) return FDKV_E_INVALID_ARG;
  fdkv_span sp{seq_lens, max_seq_len, modes, seg_offsets, cache};
  return decode_impl(dims, batch, 1, &sp, nullptr, layer, q, nullptr, sm_scale, ws, ws_bytes, stream, kPhaseSplit);
}

fdkv_status fdkv_decode_combine(const fdkv_dims* dims, int32_t batch, int32_t n_chunks, void* out, const void* ws,
                                size_t ws_bytes, void* stream) {
  fdkv_status st = check_dims(dims);
  if (st != FDKV_OK) return st;
  if (batch < 1 || n_chunks < 1 || !aligned(out, 16) || !aligned(ws, 16)) return FDKV_E_INVALID_ARG;
  const uint64_t G = dims->n_q_heads / dims->n_kv_heads;
  const uint64_t need = (uint64_t)batch * dims->n_kv_heads * n_chunks * G * (dims->head_dim + 4) * 4;
  if (ws_bytes < need) return FDKV_E_WORKSPACE;
  DecodeParams p{};
  p.out = out;
  p.ws = static_cast<float*>(const_cast<void*>(ws));
  p.hkv = dims->n_kv_heads;
  p.hq = dims->n_q_heads;
  p.d = dims->head_dim;
  p.batch = batch;
  p.bf16 = dims->dtype != FDKV_F32;
  p.n_chunks_total = n_chunks;
  const hipError_t e = launch_decode_merge(p, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "decode_merge");
  return FDKV_OK;
}

fdkv_status fdkv_decode_attn(const fdkv_dims* dims, int32_t batch, const int32_t* seq_lens, int32_t max_seq_len,
                             const uint8_t* modes, const uint64_t* seg_offsets, const void* cache, int32_t layer,
                             const void* q, void* out, float sm_scale, void* ws, size_t ws_bytes, void* stream) {
  fdkv_status st = check_dims(dims);
  if (st != FDKV_OK) return st;
  if (max_seq_len < 0) return FDKV_E_INVALID_ARG;
  fdkv_span sp{seq_lens, max_seq_len, modes, seg_offsets, cache};
  return fdkv_decode_spans(dims, batch, 1, &sp, nullptr, layer, q, out, sm_scale, ws, ws_bytes, stream);
}

size_t fdkv_decode_static_scratch_bytes(void) { return kStaticScratchBytes; }

fdkv_status fdkv_decode_attn_static(const fdkv_dims* dims, int32_t batch, const int32_t* seq_lens,
                                    int32_t max_seq_len, const uint8_t* modes, const uint64_t* seg_offsets,
                                    const void* cache, int32_t layer, const void* q, void* out, float sm_scale,
                                    void* stream) {
  fdkv_status st = check_dims(dims);
  if (st != FDKV_OK) return st;
  if (max_seq_len < 0) return FDKV_E_INVALID_ARG;
  size_t need = 0;
  st = fdkv_decode_workspace(dims, batch, max_seq_len, &need);
  if (st != FDKV_OK) return st;
  if (need > kStaticScratchBytes) {
    g_last_error = "fdkv_decode_attn_static: this call needs " + std::to_string(need) +
                   " bytes of split-K records; the static scratch holds " + std::to_string(kStaticScratchBytes);
    return FDKV_E_WORKSPACE;
  }
  void* ws = nullptr;
  st = scratch_of_current_device(&ws);
  if (st != FDKV_OK) return st;
  return fdkv_decode_attn(dims, batch, seq_lens, max_seq_len, modes, seg_offsets, cache, layer, q, out, sm_scale, ws,
                          kStaticScratchBytes, stream);
}

}  // extern "C"
