// extern "C" entry points of libwitcert: argument checks, launch shapes.
// Every entry point validates on the host, enqueues on the caller's stream and
// returns; nothing allocates, synchronizes or reads device memory back.
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <atomic>

#include "wc_launch.h"

namespace {

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

int elem_bytes(int kind) { return kind == WC_KIND_BF16 ? 2 : 1; }

// need_witness: also a BF16 cache must carry one; witness_optional: a quantized
// cache may come without one (the Tier-B decode reads none).
int check_cache(const wc_cache* c, bool need_witness, bool witness_optional = false) {
  if (c == nullptr) return WC_EINVAL;
  if (c->kind < WC_KIND_INT8_DITHER || c->kind > WC_KIND_BF16) return WC_EINVAL;
  if (c->head_dim != 64 && c->head_dim != 128) return WC_EUNSUPPORTED;
  if (c->n_kv_heads < 1 || c->n_kv_heads > 65535 || c->layer < 0 || c->layer > 65535) return WC_EINVAL;
  if (c->rope_layout != WC_ROPE_HALF && c->rope_layout != WC_ROPE_INTERLEAVED) return WC_EINVAL;
  if (c->num_blocks < 1 || !c->k_data || !c->v_data) return WC_EINVAL;
  if (!aligned16(c->k_data) || !aligned16(c->v_data)) return WC_EINVAL;
  if (c->kind != WC_KIND_BF16 || need_witness) {
    if (c->n_bands < 1 || c->n_bands > 16 || c->head_dim % (2 * c->n_bands)) return WC_EINVAL;
    if (c->k_witness ? !aligned16(c->k_witness) : !witness_optional) return WC_EINVAL;
  }
  if (c->kind == WC_KIND_INT8_DITHER &&
      (!c->k_scale || !c->v_scale || !aligned16(c->k_scale) || !aligned16(c->v_scale)))
    return WC_EINVAL;
  if (c->n_outlier_pairs != 0) {   // bypassed pairs: INT8 keys only, m even, <= 16
    const int m = c->n_outlier_pairs;
    if (c->kind != WC_KIND_INT8_DITHER || m < 0 || m > 16 || (m & 1) || m > c->head_dim / 2)
      return WC_EINVAL;
    if (!c->outlier_pairs || !c->k_outlier || !aligned16(c->k_outlier)) return WC_EINVAL;
  }
  if ((c->v_resid != nullptr) != (c->v_norm != nullptr)) return WC_EINVAL;   // value side: both or neither
  if (c->v_resid != nullptr &&
      (c->kind == WC_KIND_BF16 || !aligned16(c->v_resid) || !aligned16(c->v_norm)))
    return WC_EINVAL;
  if (c->group_scales != 0 && (c->group_scales != 1 || c->kind != WC_KIND_INT8_DITHER)) return WC_EINVAL;
  // persistent repair marks: quantized kinds, with the exact store's pages
  if (c->repaired != nullptr &&
      (c->kind == WC_KIND_BF16 || !c->exact_k || !c->exact_v || !aligned16(c->exact_k) || !aligned16(c->exact_v)))
    return WC_EINVAL;
  return WC_OK;
}

int hip_status(hipError_t e) { return e == hipSuccess ? WC_OK : WC_EHIP; }

// Scratch of wc_step_metered_decode_gate_noalloc (the decode's split records and
// gate counters) for callers that cannot allocate: a fixed array in device
// memory, one copy per GPU, held until the process ends.  In host code `scratch`
// names a host-side stand-in, never the device memory: kernels get the address
// hipGetSymbolAddress returns on each device, looked up once per device on its
// first use there (with that device current) and kept in scratch_dev.
__device__ __attribute__((aligned(256))) uint8_t scratch[WC_NOALLOC_SCRATCH_BYTES];
constexpr int kMaxDevices = 64;
std::atomic<void*> scratch_dev[kMaxDevices];

int scratch_address(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return WC_EHIP;
  if (dev >= kMaxDevices) return WC_EUNSUPPORTED;
  void* p = scratch_dev[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return WC_EHIP;
    scratch_dev[dev].store(p, std::memory_order_release);
  }
  *out = p;
  return WC_OK;
}

}  // namespace

extern "C" {

const char* wc_strerror(int status) {
  switch (status) {
    case WC_OK: return "ok";
    case WC_EINVAL: return "invalid argument";
    case WC_EUNSUPPORTED: return "unsupported configuration";
    case WC_EHIP: return "HIP launch error";
    case WC_EWORKSPACE: return "workspace too small";
    case WC_ESCRATCH: return "sizes exceed the static scratch of the no-allocation entry point";
    default: return "unknown status";
  }
}

int wc_version(void) { return 106; }   // 1.6: the speculative step's split query

size_t wc_cache_bytes(int kind, int64_t num_blocks, int n_kv_heads, int head_dim, int n_bands,
                      int n_outlier_pairs, int value_side, int group_scales, size_t sizes[8]) {
  if (kind < WC_KIND_INT8_DITHER || kind > WC_KIND_BF16 || num_blocks < 0 || n_kv_heads < 1 ||
      head_dim < 1 || (kind != WC_KIND_BF16 && n_bands < 1))
    return 0;
  if (n_outlier_pairs < 0 || n_outlier_pairs > 16 || (n_outlier_pairs & 1) ||
      2 * n_outlier_pairs > head_dim || (n_outlier_pairs && kind != WC_KIND_INT8_DITHER))
    return 0;
  if (value_side && kind == WC_KIND_BF16) return 0;
  if (group_scales && (kind != WC_KIND_INT8_DITHER || head_dim % 32)) return 0;
  const size_t slots = (size_t)num_blocks * WC_BLOCK_TOKENS * (size_t)n_kv_heads;
  size_t s[8];
  s[0] = s[1] = slots * head_dim * elem_bytes(kind);
  // one fp16 scale per token, or per 32-channel group (Table 4)
  s[2] = s[3] = kind == WC_KIND_INT8_DITHER ? slots * 2 * (group_scales ? head_dim / 32 : 1) : 0;
  s[4] = kind == WC_KIND_BF16 ? 0 : slots * n_bands * 2;
  s[5] = slots * (size_t)n_outlier_pairs * 4;   // 2m fp16 values per token-head
  s[6] = s[7] = value_side ? slots * 2 : 0;     // value residual, value norm
  if (sizes) memcpy(sizes, s, sizeof(s));
  size_t total = 0;
  for (size_t x : s) total += x;
  return total;
}

// The write's arguments after its checks (WC_OK with a.n_tok == 0: nothing to do).
static int write_args(const wc_cache* cache, const wc_cache* exact, const void* k, const void* v,
                      int in_dtype, const int64_t* slot_mapping, int64_t n_tok, wc::WriteArgs& a) {
  a = wc::WriteArgs{};
  int st = check_cache(cache, false);
  if (st != WC_OK) return st;
  if (exact != nullptr) {
    st = check_cache(exact, false);
    if (st != WC_OK) return st;
    if (cache->kind == WC_KIND_BF16 || exact->kind != WC_KIND_BF16 ||
        exact->head_dim != cache->head_dim || exact->n_kv_heads != cache->n_kv_heads ||
        exact->num_blocks < cache->num_blocks)
      return WC_EINVAL;
  }
  if (n_tok < 0 || (in_dtype != WC_F32 && in_dtype != WC_BF16)) return WC_EINVAL;
  if (n_tok == 0) return WC_OK;
  if (!k || !v || !slot_mapping || !aligned16(k) || !aligned16(v)) return WC_EINVAL;
  a.kind = cache->kind;
  a.head_dim = cache->head_dim;
  a.n_kv = cache->n_kv_heads;
  a.n_bands = cache->n_bands;
  a.interleaved = cache->rope_layout == WC_ROPE_INTERLEAVED;
  a.layer = cache->layer;
  a.in_dtype = in_dtype;
  a.key0 = (uint32_t)cache->seed;
  a.key1 = (uint32_t)(cache->seed >> 32);
  a.n_tok = n_tok;
  a.n_slots = cache->num_blocks * WC_BLOCK_TOKENS;   // (an exact copy has at least as many blocks)
  a.k = k;
  a.v = v;
  a.slots = slot_mapping;
  a.k_data = cache->k_data;
  a.v_data = cache->v_data;
  a.k_scale = static_cast<uint16_t*>(cache->k_scale);
  a.v_scale = static_cast<uint16_t*>(cache->v_scale);
  a.k_witness = static_cast<uint16_t*>(cache->k_witness);
  a.x_k_data = exact ? exact->k_data : nullptr;
  a.x_v_data = exact ? exact->v_data : nullptr;
  a.n_pairs = cache->n_outlier_pairs;
  a.pairs = cache->outlier_pairs;
  a.k_outlier = static_cast<uint16_t*>(cache->k_outlier);
  a.v_resid = static_cast<uint16_t*>(cache->v_resid);
  a.v_norm = static_cast<uint16_t*>(cache->v_norm);
  a.group_scales = cache->group_scales;
  return WC_OK;
}

static int write_common(const wc_cache* cache, const wc_cache* exact, const void* k, const void* v,
                        int in_dtype, const int64_t* slot_mapping, int64_t n_tok, void* stream) {
  wc::WriteArgs a;
  const int st = write_args(cache, exact, k, v, in_dtype, slot_mapping, n_tok, a);
  if (st != WC_OK || a.n_tok == 0) return st;
  return hip_status(wc::launch_quantize_write(a, static_cast<hipStream_t>(stream)));
}

int wc_quantize_write(const wc_cache* cache, const void* k, const void* v, int in_dtype,
                      const int64_t* slot_mapping, int64_t n_tok, void* stream) {
  return write_common(cache, nullptr, k, v, in_dtype, slot_mapping, n_tok, stream);
}

int wc_quantize_write_pair(const wc_cache* cache, const wc_cache* exact, const void* k, const void* v,
                           int in_dtype, const int64_t* slot_mapping, int64_t n_tok, void* stream) {
  if (exact == nullptr) return WC_EINVAL;
  return write_common(cache, exact, k, v, in_dtype, slot_mapping, n_tok, stream);
}

int wc_witness(const void* x, int x_dtype, const void* xhat, int xhat_dtype, int64_t n_vec,
               int head_dim, int n_bands, int rope_layout, uint16_t* w_out, void* stream) {
  if (n_vec < 0 || head_dim < 2 || n_bands < 1 || n_bands > 64 || head_dim % (2 * n_bands))
    return WC_EINVAL;
  if (x_dtype < WC_F32 || x_dtype > WC_F16 || xhat_dtype < WC_F32 || xhat_dtype > WC_F16)
    return WC_EINVAL;
  if (rope_layout != WC_ROPE_HALF && rope_layout != WC_ROPE_INTERLEAVED) return WC_EINVAL;
  if (n_vec == 0) return WC_OK;
  if (!x || !xhat || !w_out) return WC_EINVAL;
  wc::WitnessArgs a{x, xhat, x_dtype, xhat_dtype, head_dim, n_bands,
                    rope_layout == WC_ROPE_INTERLEAVED, n_vec, w_out};
  return hip_status(wc::launch_witness(a, static_cast<hipStream_t>(stream)));
}

size_t wc_select_workspace_size(int64_t n_tok, int n_kv_heads, int head_dim) {
  if (n_tok < 1 || n_kv_heads < 1 || head_dim < 2) return 0;
  return (size_t)n_kv_heads * wc::select_chunks(n_tok) * (head_dim / 2) * sizeof(double);
}

int wc_select_outlier_pairs(const void* k, int in_dtype, int64_t n_tok, int n_kv_heads,
                            int head_dim, int rope_layout, int m, int32_t* pairs_out, void* ws,
                            size_t ws_bytes, void* stream) {
  if (n_tok < 1 || n_kv_heads < 1 || n_kv_heads > 65535 || (in_dtype != WC_F32 && in_dtype != WC_BF16))
    return WC_EINVAL;
  if (head_dim != 64 && head_dim != 128) return WC_EUNSUPPORTED;
  if (rope_layout != WC_ROPE_HALF && rope_layout != WC_ROPE_INTERLEAVED) return WC_EINVAL;
  if (m < 0 || m > head_dim / 2) return WC_EINVAL;
  if (m == 0) return WC_OK;
  if (!k || !pairs_out || !ws || !aligned16(k) || ((uintptr_t)ws & 7u)) return WC_EINVAL;
  if (ws_bytes < wc_select_workspace_size(n_tok, n_kv_heads, head_dim)) return WC_EWORKSPACE;
  wc::SelectArgs a{};
  a.k = k;
  a.in_dtype = in_dtype;
  a.n_kv = n_kv_heads;
  a.head_dim = head_dim;
  a.interleaved = rope_layout == WC_ROPE_INTERLEAVED;
  a.m = m;
  a.n_chunks = wc::select_chunks(n_tok);
  a.n_tok = n_tok;
  a.pairs_out = pairs_out;
  a.part = static_cast<double*>(ws);
  return hip_status(wc::launch_select_pairs(a, static_cast<hipStream_t>(stream)));
}

size_t wc_decode_workspace_size(int batch, int n_q_heads, int n_kv_heads, int head_dim,
                                int64_t max_seq_len, int split_tokens) {
  if (batch < 0 || n_q_heads < 1 || n_kv_heads < 1 || head_dim < 1 || max_seq_len < 0 ||
      split_tokens < 0)
    return 0;
  const int st = wc::choose_split_tokens(batch, n_kv_heads, max_seq_len, split_tokens);
  const int64_t ns = wc::n_splits_for(max_seq_len, st);
  return wc::records_bytes(batch, n_q_heads, ns, head_dim) + wc::gate_unit_bytes(batch, n_kv_heads) +
         wc::share_bytes(batch, n_q_heads, ns, st);
}

int wc_decode_split_tokens(int batch, int n_kv_heads, int64_t max_seq_len, int64_t total_tokens,
                           int split_tokens) {
  if (batch < 0 || n_kv_heads < 1 || max_seq_len < 0 || total_tokens < 0 || split_tokens < 0) return 0;
  if (split_tokens > 0 || total_tokens == 0)
    return wc::choose_split_tokens(batch, n_kv_heads, max_seq_len, split_tokens);
  return wc::choose_split_tokens_total(n_kv_heads, max_seq_len, total_tokens);
}

int wc_speculative_split_tokens(int batch, int n_kv_heads, int64_t max_seq_len, int64_t total_tokens,
                                int split_tokens) {
  if (batch < 0 || n_kv_heads < 1 || max_seq_len < 0 || total_tokens < 0 || split_tokens < 0) return 0;
  const int64_t target = wc::kDecodeWorkgroups / 2;
  if (split_tokens > 0 || total_tokens == 0)
    return wc::choose_split_tokens(batch, n_kv_heads, max_seq_len, split_tokens, target);
  return wc::choose_split_tokens_total(n_kv_heads, max_seq_len, total_tokens, target);
}

static int decode_common(const wc_cache* cache, const void* q, int q_dtype, int batch,
                         int n_q_heads, const int32_t* block_table, int max_blocks_per_seq,
                         const int32_t* seq_lens, int64_t max_seq_len, float sm_scale, void* out,
                         int out_dtype, int split_tokens, void* ws, size_t ws_bytes,
                         wc::DecodeArgs& a) {
  if (batch < 0 || n_q_heads < 1 || max_blocks_per_seq < 1 || max_seq_len < 0 || split_tokens < 0)
    return WC_EINVAL;
  if (n_q_heads % cache->n_kv_heads) return WC_EINVAL;
  const int group = n_q_heads / cache->n_kv_heads;
  if (group > 16) return WC_EUNSUPPORTED;
  if (q_dtype != WC_F32 && q_dtype != WC_BF16) return WC_EINVAL;
  if (out_dtype != WC_F32 && out_dtype != WC_BF16) return WC_EINVAL;
  if (max_seq_len > (int64_t)max_blocks_per_seq * WC_BLOCK_TOKENS || max_seq_len > INT32_MAX / 2)
    return WC_EINVAL;
  if (!(sm_scale > 0.0f)) return WC_EINVAL;
  if (batch > 0 && (!q || !block_table || !seq_lens || !out || !ws)) return WC_EINVAL;
  const int st = wc::choose_split_tokens(batch, cache->n_kv_heads, max_seq_len, split_tokens);
  const int64_t ns = wc::n_splits_for(max_seq_len, st);
  if (ns > 65535) return WC_EUNSUPPORTED;
  if (ws_bytes < wc_decode_workspace_size(batch, n_q_heads, cache->n_kv_heads, cache->head_dim,
                                          max_seq_len, split_tokens))
    return WC_EWORKSPACE;
  a.k_data = cache->k_data;
  a.v_data = cache->v_data;
  a.k_scale = static_cast<const uint16_t*>(cache->k_scale);
  a.v_scale = static_cast<const uint16_t*>(cache->v_scale);
  a.k_witness = static_cast<const uint16_t*>(cache->k_witness);
  a.q = q;
  a.table = block_table;
  a.seq_lens = seq_lens;
  a.num_blocks = cache->num_blocks;
  a.part = static_cast<float*>(ws);
  a.gate_unit = reinterpret_cast<int32_t*>(static_cast<char*>(ws) +
                                           wc::records_bytes(batch, n_q_heads, ns, cache->head_dim));
  a.shares = reinterpret_cast<float4*>(static_cast<char*>(ws) +
                                       wc::records_bytes(batch, n_q_heads, ns, cache->head_dim) +
                                       wc::gate_unit_bytes(batch, cache->n_kv_heads));
  a.share_slots = wc::share_slots(st);
  a.out = out;
  a.kind = cache->kind;
  a.head_dim = cache->head_dim;
  a.n_bands = cache->n_bands;
  a.interleaved = cache->rope_layout == WC_ROPE_INTERLEAVED;
  a.q_dtype = q_dtype;
  a.out_dtype = out_dtype;
  a.batch = batch;
  a.n_q = n_q_heads;
  a.n_kv = cache->n_kv_heads;
  a.group = group;
  a.max_blocks = max_blocks_per_seq;
  a.n_splits = (int)ns;
  a.split_tokens = st;
  a.layer = cache->layer;
  a.key0 = (uint32_t)cache->seed;
  a.key1 = (uint32_t)(cache->seed >> 32);
  a.sm_scale = sm_scale;
  a.n_pairs = cache->n_outlier_pairs;
  a.pairs = cache->outlier_pairs;
  a.k_outlier = static_cast<const uint16_t*>(cache->k_outlier);
  a.v_resid = static_cast<const uint16_t*>(cache->v_resid);
  a.v_norm = static_cast<const uint16_t*>(cache->v_norm);
  a.group_scales = cache->group_scales;
  a.repaired = cache->repaired;
  a.x_k_data = cache->repaired ? cache->exact_k : nullptr;
  a.x_v_data = cache->repaired ? cache->exact_v : nullptr;
  // WITCERT_FORCE_VALU=1 selects the vector-ALU kernels even where the
  // matrix-core ones apply (used to cross-check the two paths)
  const char* force = getenv("WITCERT_FORCE_VALU");
  a.use_mfma = !(force && force[0] == '1');
  return WC_OK;
}

int wc_metered_decode_attention(const wc_cache* cache, const void* q, int q_dtype, int batch,
                                int n_q_heads, const int32_t* block_table,
                                int max_blocks_per_seq, const int32_t* seq_lens,
                                int64_t max_seq_len, float sm_scale, void* out, int out_dtype,
                                float* meter, float* raw, int split_tokens, void* ws,
                                size_t ws_bytes, void* stream) {
  int s = check_cache(cache, true);
  if (s != WC_OK) return s;
  if (cache->kind == WC_KIND_BF16) return WC_EINVAL;
  if (batch > 0 && !meter) return WC_EINVAL;
  wc::DecodeArgs a{};
  s = decode_common(cache, q, q_dtype, batch, n_q_heads, block_table, max_blocks_per_seq,
                    seq_lens, max_seq_len, sm_scale, out, out_dtype, split_tokens, ws, ws_bytes, a);
  if (s != WC_OK) return s;
  a.meter = meter;
  a.raw = raw;
  a.mask_kv = nullptr;
  return hip_status(wc::launch_decode(a, true, static_cast<hipStream_t>(stream)));
}

double wc_tierb_delta_loc(double delta_req, int n_layers, int n_q_heads, int n_steps) {
  if (!(delta_req > 0.0 && delta_req < 1.0) || n_layers < 1 || n_q_heads < 1 || n_steps < 1) return -1.0;
  return delta_req / ((double)n_layers * (double)n_q_heads * (double)n_steps);
}

int wc_tierb_decode_attention(const wc_cache* cache, const void* q, int q_dtype, int batch,
                              int n_q_heads, const int32_t* block_table, int max_blocks_per_seq,
                              const int32_t* seq_lens, int64_t max_seq_len, float sm_scale,
                              void* out, int out_dtype, float* meter, float* raw, int split_tokens,
                              float delta_loc, void* ws, size_t ws_bytes, void* stream) {
  int s = check_cache(cache, false, true);   // no witness is read
  if (s != WC_OK) return s;
  if (cache->kind != WC_KIND_INT8_DITHER) return WC_EINVAL;
  if (!(delta_loc > 0.0f && delta_loc < 1.0f)) return WC_EINVAL;
  if (batch > 0 && !meter) return WC_EINVAL;
  wc::DecodeArgs a{};
  s = decode_common(cache, q, q_dtype, batch, n_q_heads, block_table, max_blocks_per_seq,
                    seq_lens, max_seq_len, sm_scale, out, out_dtype, split_tokens, ws, ws_bytes, a);
  if (s != WC_OK) return s;
  a.meter = meter;
  a.raw = raw;
  a.tierb_delta = delta_loc;
  return hip_status(wc::launch_decode(a, true, static_cast<hipStream_t>(stream)));
}

int wc_metered_decode_gate(const wc_cache* cache, const void* q, int q_dtype, int batch,
                           int n_q_heads, const int32_t* block_table, int max_blocks_per_seq,
                           const int32_t* seq_lens, int64_t max_seq_len, float sm_scale, void* out,
                           int out_dtype, float* meter, float* raw, int split_tokens, float tau,
                           uint8_t* mask_q, uint8_t* mask_kv, int32_t* n_gated, void* ws,
                           size_t ws_bytes, void* stream) {
  int s = check_cache(cache, true);
  if (s != WC_OK) return s;
  if (cache->kind == WC_KIND_BF16) return WC_EINVAL;
  if (!(tau >= 0.0f)) return WC_EINVAL;
  if (batch > 0 && (!meter || !mask_q || !mask_kv)) return WC_EINVAL;
  wc::DecodeArgs a{};
  s = decode_common(cache, q, q_dtype, batch, n_q_heads, block_table, max_blocks_per_seq,
                    seq_lens, max_seq_len, sm_scale, out, out_dtype, split_tokens, ws, ws_bytes, a);
  if (s != WC_OK) return s;
  a.meter = meter;
  a.raw = raw;
  a.gate_mask_q = mask_q;
  a.gate_mask_kv = mask_kv;
  a.gate_count = n_gated;
  a.gate_tau = tau;
  return hip_status(wc::launch_decode(a, true, static_cast<hipStream_t>(stream)));
}

static int step_common(const wc_cache* cache, const wc_cache* exact, const void* new_k,
                       const void* new_v, int in_dtype, const int64_t* new_slots, const void* q,
                       int q_dtype, int batch, int n_q_heads, const int32_t* block_table,
                       int max_blocks_per_seq, const int32_t* seq_lens, int64_t max_seq_len,
                       float sm_scale, void* out, int out_dtype, float* meter, float* raw,
                       int split_tokens, float tau, uint8_t* mask_q, uint8_t* mask_kv,
                       int32_t* n_gated, void* ws, size_t ws_bytes, void* stream) {
  if (exact == nullptr) return WC_EINVAL;
  wc::WriteArgs w;
  int s = write_args(cache, exact, new_k, new_v, in_dtype, new_slots, batch, w);
  if (s != WC_OK) return s;
  s = check_cache(cache, true);
  if (s != WC_OK) return s;
  if (cache->kind == WC_KIND_BF16) return WC_EINVAL;
  if (!(tau >= 0.0f)) return WC_EINVAL;
  if (batch > 0 && (!meter || !mask_q || !mask_kv)) return WC_EINVAL;
  wc::DecodeArgs a{};
  s = decode_common(cache, q, q_dtype, batch, n_q_heads, block_table, max_blocks_per_seq,
                    seq_lens, max_seq_len, sm_scale, out, out_dtype, split_tokens, ws, ws_bytes, a);
  if (s != WC_OK) return s;
  a.meter = meter;
  a.raw = raw;
  a.gate_mask_q = mask_q;
  a.gate_mask_kv = mask_kv;
  a.gate_count = n_gated;
  a.gate_tau = tau;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  if (batch == 0) return WC_OK;
  if (wc::step_write_fusable(a) && in_dtype == WC_BF16) {
    // one launch: the workgroup holding a sequence's new token writes it first
    a.sw = w;
    a.step_write = 1;
    return hip_status(wc::launch_decode(a, true, st));
  }
  const hipError_t e = wc::launch_quantize_write(w, st);
  return hip_status(e != hipSuccess ? e : wc::launch_decode(a, true, st));
}

int wc_step_metered_decode_gate(const wc_cache* cache, const wc_cache* exact, const void* new_k,
                                const void* new_v, int in_dtype, const int64_t* new_slots, const void* q,
                                int q_dtype, int batch, int n_q_heads, const int32_t* block_table,
                                int max_blocks_per_seq, const int32_t* seq_lens, int64_t max_seq_len,
                                float sm_scale, void* out, int out_dtype, float* meter, float* raw,
                                int split_tokens, float tau, uint8_t* mask_q, uint8_t* mask_kv,
                                int32_t* n_gated, void* ws, size_t ws_bytes, void* stream) {
  return step_common(cache, exact, new_k, new_v, in_dtype, new_slots, q, q_dtype, batch, n_q_heads,
                     block_table, max_blocks_per_seq, seq_lens, max_seq_len, sm_scale, out, out_dtype, meter,
                     raw, split_tokens, tau, mask_q, mask_kv, n_gated, ws, ws_bytes, stream);
}

int wc_step_metered_decode_gate_noalloc(const wc_cache* cache, const wc_cache* exact, const void* new_k,
                                        const void* new_v, int in_dtype, const int64_t* new_slots,
                                        const void* q, int q_dtype, int batch, int n_q_heads,
                                        const int32_t* block_table, int max_blocks_per_seq,
                                        const int32_t* seq_lens, int64_t max_seq_len, float sm_scale,
                                        void* out, int out_dtype, float* meter, float* raw, int split_tokens,
                                        float tau, uint8_t* mask_q, uint8_t* mask_kv, int32_t* n_gated,
                                        void* stream) {
  if (cache == nullptr) return WC_EINVAL;
  // (a size of 0 means invalid sizes: step_common reports those)
  const size_t need = wc_decode_workspace_size(batch, n_q_heads, cache->n_kv_heads, cache->head_dim,
                                               max_seq_len, split_tokens);
  if (need > (size_t)WC_NOALLOC_SCRATCH_BYTES) return WC_ESCRATCH;
  void* ws = nullptr;
  const int s = scratch_address(&ws);
  if (s != WC_OK) return s;
  return step_common(cache, exact, new_k, new_v, in_dtype, new_slots, q, q_dtype, batch, n_q_heads,
                     block_table, max_blocks_per_seq, seq_lens, max_seq_len, sm_scale, out, out_dtype, meter,
                     raw, split_tokens, tau, mask_q, mask_kv, n_gated, ws, (size_t)WC_NOALLOC_SCRATCH_BYTES,
                     stream);
}

size_t wc_certified_workspace_size(int batch, int n_q_heads, int n_kv_heads, int head_dim, int64_t max_seq_len,
                                   int split_tokens) {
  const size_t base = wc_decode_workspace_size(batch, n_q_heads, n_kv_heads, head_dim, max_seq_len, split_tokens);
  if (base == 0) return 0;
  const int st = wc::choose_split_tokens(batch, n_kv_heads, max_seq_len, split_tokens);
  return base + wc::records_bytes(batch, n_q_heads, wc::n_splits_for(max_seq_len, st), head_dim);
}

// Certified step: the step write and the metered decode (records in the first
// region of the workspace; no block segments: this call repairs nothing), the
// exact fallback with the gate decided in its prologue from those records
// (records in the second region), the final merge.
// The certified step (spec = false: the exact fallback decides each unit's gate in
// its prologue and reads the routed units) or its speculative form (spec = true:
// the exact fallback of every unit runs beside the metered decode, in one launch
// where the kernels allow it, and the final merge decides the gates).
static int certified_step(const wc_cache* cache, const wc_cache* exact, const void* new_k, const void* new_v,
                          int in_dtype, const int64_t* new_slots, const void* q, int q_dtype, int batch,
                          int n_q_heads, const int32_t* block_table, int max_blocks_per_seq,
                          const int32_t* seq_lens, int64_t max_seq_len, float sm_scale, void* out, int out_dtype,
                          float* meter, float* raw, int split_tokens, float tau, uint8_t* mask_q, uint8_t* mask_kv,
                          int32_t* n_gated, void* ws, size_t ws_bytes, void* stream, bool spec) {
  if (cache == nullptr || exact == nullptr) return WC_EINVAL;
  wc::WriteArgs w;
  int s = write_args(cache, exact, new_k, new_v, in_dtype, new_slots, batch, w);
  if (s != WC_OK) return s;
  s = check_cache(cache, true);
  if (s != WC_OK) return s;
  s = check_cache(exact, false);
  if (s != WC_OK) return s;
  if (cache->kind == WC_KIND_BF16 || exact->kind != WC_KIND_BF16) return WC_EINVAL;
  if (exact->n_kv_heads != cache->n_kv_heads || exact->head_dim != cache->head_dim) return WC_EINVAL;
  if (!(tau >= 0.0f)) return WC_EINVAL;
  if (batch > 0 && (!meter || !mask_q || !mask_kv)) return WC_EINVAL;
  if (n_q_heads < 1 || split_tokens < 0 || max_seq_len < 0 || batch < 0) return WC_EINVAL;
  const size_t need = wc_certified_workspace_size(batch, n_q_heads, cache->n_kv_heads, cache->head_dim,
                                                  max_seq_len, split_tokens);
  if (need == 0) return WC_EINVAL;
  if (ws_bytes < need) return WC_EWORKSPACE;
  const int st = wc::choose_split_tokens(batch, cache->n_kv_heads, max_seq_len, split_tokens);
  const size_t rb = wc::records_bytes(batch, n_q_heads, wc::n_splits_for(max_seq_len, st), cache->head_dim);
  char* wsb = static_cast<char*>(ws);
  wc::DecodeArgs am{}, ax{};
  s = decode_common(cache, q, q_dtype, batch, n_q_heads, block_table, max_blocks_per_seq, seq_lens, max_seq_len,
                    sm_scale, out, out_dtype, split_tokens, wsb, ws_bytes, am);
  if (s != WC_OK) return s;
  s = decode_common(exact, q, q_dtype, batch, n_q_heads, block_table, max_blocks_per_seq, seq_lens, max_seq_len,
                    sm_scale, out, out_dtype, split_tokens, wsb + rb, ws_bytes - rb, ax);
  if (s != WC_OK) return s;
  // (the metered call's gate counters and block segments would overlap the second
  // region: neither is used here)
  am.shares = nullptr;
  am.gate_unit = nullptr;
  if (batch == 0) return WC_OK;
  const hipStream_t hs = static_cast<hipStream_t>(stream);
  am.no_merge = 1;
  ax.no_merge = 1;
  hipError_t e = hipSuccess;
  const bool fuse_write = wc::step_write_fusable(am) && in_dtype == WC_BF16;
  if (spec && wc::spec_decode_fusable(am, ax)) {
    // 1-2. one launch: the metered decode and the exact fallback of every unit, each
    //      writing the step's tokens into the cache it reads first
    if (fuse_write) {
      wc::WriteArgs wx;
      s = write_args(cache, nullptr, new_k, new_v, in_dtype, new_slots, batch, am.sw);
      if (s == WC_OK) s = write_args(exact, nullptr, new_k, new_v, in_dtype, new_slots, batch, wx);
      if (s != WC_OK) return s;
      am.step_write = 1;
      ax.sw = wx;
      ax.step_write = 1;
    } else {
      e = wc::launch_quantize_write(w, hs);
    }
    if (e == hipSuccess) e = wc::launch_decode_spec(am, ax, hs);
  } else {
    // 1. the metered decode (with the step's tokens written first), no merge
    if (fuse_write) {
      am.sw = w;
      am.step_write = 1;
    } else {
      e = wc::launch_quantize_write(w, hs);
    }
    if (e == hipSuccess) e = wc::launch_decode(am, true, hs);
    // 2. the exact fallback: each unit's gate from the metered records, then the
    //    routed units' exact records (speculative: every unit's, no gate)
    if (!spec) {
      ax.gate_part = am.part;
      ax.gate_tau = tau;
      ax.gate_mask_q = mask_q;
      ax.gate_mask_kv = mask_kv;
    }
    if (e == hipSuccess) e = wc::launch_decode(ax, false, hs);
  }
  // 3. the final merge: routed heads from the exact records, the others from the
  //    metered ones; meter and raw from the metered records (speculative: the merge
  //    decides the gates from the metered records)
  wc::DecodeArgs af = am;
  af.step_write = 0;
  af.no_merge = 0;
  af.x_part = ax.part;
  af.meter = meter;
  af.raw = raw;
  af.gate_mask_q = mask_q;
  af.gate_mask_kv = mask_kv;
  af.gate_count = n_gated;
  af.gate_tau = tau;
  if (spec) {
    af.gate_part = am.part;
    af.merge_gate = 1;
  }
  if (e == hipSuccess) e = wc::launch_merge(af, true, hs);
  return hip_status(e);
}

int wc_step_certified_decode(const wc_cache* cache, const wc_cache* exact, const void* new_k, const void* new_v,
                             int in_dtype, const int64_t* new_slots, const void* q, int q_dtype, int batch,
                             int n_q_heads, const int32_t* block_table, int max_blocks_per_seq,
                             const int32_t* seq_lens, int64_t max_seq_len, float sm_scale, void* out,
                             int out_dtype, float* meter, float* raw, int split_tokens, float tau, uint8_t* mask_q,
                             uint8_t* mask_kv, int32_t* n_gated, void* ws, size_t ws_bytes, void* stream) {
  return certified_step(cache, exact, new_k, new_v, in_dtype, new_slots, q, q_dtype, batch, n_q_heads, block_table,
                        max_blocks_per_seq, seq_lens, max_seq_len, sm_scale, out, out_dtype, meter, raw,
                        split_tokens, tau, mask_q, mask_kv, n_gated, ws, ws_bytes, stream, false);
}

int wc_step_certified_decode_speculative(const wc_cache* cache, const wc_cache* exact, const void* new_k,
                                         const void* new_v, int in_dtype, const int64_t* new_slots, const void* q,
                                         int q_dtype, int batch, int n_q_heads, const int32_t* block_table,
                                         int max_blocks_per_seq, const int32_t* seq_lens, int64_t max_seq_len,
                                         float sm_scale, void* out, int out_dtype, float* meter, float* raw,
                                         int split_tokens, float tau, uint8_t* mask_q, uint8_t* mask_kv,
                                         int32_t* n_gated, void* ws, size_t ws_bytes, void* stream) {
  return certified_step(cache, exact, new_k, new_v, in_dtype, new_slots, q, q_dtype, batch, n_q_heads, block_table,
                        max_blocks_per_seq, seq_lens, max_seq_len, sm_scale, out, out_dtype, meter, raw,
                        split_tokens, tau, mask_q, mask_kv, n_gated, ws, ws_bytes, stream, true);
}

int wc_joint_decode_gate(const wc_cache* cache, const void* q, int q_dtype, int batch,
                         int n_q_heads, const int32_t* block_table, int max_blocks_per_seq,
                         const int32_t* seq_lens, int64_t max_seq_len, float sm_scale, void* out,
                         int out_dtype, float* meter, float* raw, float* meter_v, int split_tokens,
                         float delta_loc, float tau, float tau_v, uint8_t* mask_q, uint8_t* mask_kv,
                         int32_t* n_gated, void* ws, size_t ws_bytes, void* stream) {
  const bool tierb = delta_loc != 0.0f;
  int s = check_cache(cache, !tierb, tierb);   // Tier B reads no witness
  if (s != WC_OK) return s;
  if (cache->kind == WC_KIND_BF16 || !cache->v_resid) return WC_EINVAL;
  if (tierb && (cache->kind != WC_KIND_INT8_DITHER || !(delta_loc > 0.0f && delta_loc < 1.0f)))
    return WC_EINVAL;
  if (!(tau >= 0.0f) || !(tau_v >= 0.0f)) return WC_EINVAL;
  if (batch > 0 && (!meter || !meter_v || !mask_q || !mask_kv)) return WC_EINVAL;
  wc::DecodeArgs a{};
  s = decode_common(cache, q, q_dtype, batch, n_q_heads, block_table, max_blocks_per_seq,
                    seq_lens, max_seq_len, sm_scale, out, out_dtype, split_tokens, ws, ws_bytes, a);
  if (s != WC_OK) return s;
  a.meter = meter;
  a.raw = raw;
  a.meter_v = meter_v;
  a.tierb_delta = tierb ? delta_loc : 0.0f;
  a.gate_mask_q = mask_q;
  a.gate_mask_kv = mask_kv;
  a.gate_count = n_gated;
  a.gate_tau = tau;
  a.gate_tau_v = tau_v;
  return hip_status(wc::launch_decode(a, true, static_cast<hipStream_t>(stream)));
}

int wc_block_repair(const wc_cache* cache, const wc_cache* exact, const void* q, int q_dtype,
                    int batch, int n_q_heads, const int32_t* block_table, int max_blocks_per_seq,
                    const int32_t* seq_lens, int64_t max_seq_len, float sm_scale, int split_tokens,
                    float delta_loc, float tau, int max_repair_blocks, const void* ws,
                    size_t ws_bytes, void* out, int out_dtype, float* meter, float* raw,
                    uint8_t* mask_kv, int32_t* repaired, int32_t* n_repaired, void* repair_ws,
                    size_t repair_ws_bytes, void* stream) {
  const bool tierb = delta_loc != 0.0f;
  int s = check_cache(cache, !tierb, tierb);
  if (s != WC_OK) return s;
  s = check_cache(exact, false);
  if (s != WC_OK) return s;
  if (cache->kind == WC_KIND_BF16 || exact->kind != WC_KIND_BF16 || exact->head_dim != cache->head_dim ||
      exact->n_kv_heads != cache->n_kv_heads || exact->num_blocks < cache->num_blocks)
    return WC_EINVAL;
  if (tierb && (cache->kind != WC_KIND_INT8_DITHER || !(delta_loc > 0.0f && delta_loc < 1.0f)))
    return WC_EINVAL;
  // the marked pages were served from the cache's exact store: the same cache here
  if (cache->repaired != nullptr && (cache->exact_k != exact->k_data || cache->exact_v != exact->v_data))
    return WC_EINVAL;
  if (!(tau >= 0.0f) || max_repair_blocks < 1 || max_repair_blocks > 64) return WC_EINVAL;
  if (batch > 0 && (!meter || !mask_kv)) return WC_EINVAL;
  wc::DecodeArgs a{};
  s = decode_common(cache, q, q_dtype, batch, n_q_heads, block_table, max_blocks_per_seq,
                    seq_lens, max_seq_len, sm_scale, out, out_dtype, split_tokens,
                    const_cast<void*>(ws), ws_bytes, a);   // the records are only read
  if (s != WC_OK) return s;
  if ((max_seq_len + wc::kRepairBlockTokens - 1) / wc::kRepairBlockTokens > wc::repair_max_blocks())
    return WC_EUNSUPPORTED;
  if (batch == 0) return WC_OK;
  if (!repair_ws || reinterpret_cast<uintptr_t>(repair_ws) % 256) return WC_EINVAL;
  if (repair_ws_bytes < wc_block_repair_workspace_size(batch, n_q_heads, cache->n_kv_heads,
                                                       cache->head_dim, max_repair_blocks))
    return WC_EWORKSPACE;
  a.meter = meter;
  a.raw = raw;
  a.mask_kv = mask_kv;
  a.tierb_delta = tierb ? delta_loc : 0.0f;
  wc::RepairArgs r{};
  r.d = a;
  r.d.num_blocks = exact->num_blocks < cache->num_blocks ? exact->num_blocks : cache->num_blocks;
  r.x_k_data = exact->k_data;
  r.x_v_data = exact->v_data;
  r.tau = tau;
  r.max_rep = max_repair_blocks;
  r.mask_kv_out = mask_kv;
  r.rep_list = repaired;
  r.n_rep = n_repaired;
  r.rws = repair_ws;
  // WITCERT_REPAIR_ROUND0=n caps the first round of block corrections at n blocks
  // (default: the predicted count plus one); the result does not depend on it
  const char* r0 = getenv("WITCERT_REPAIR_ROUND0");
  r.round0_cap = r0 != nullptr ? atoi(r0) : 0;
  r.tiles = wc::kRepairTiles;
  r.unit_bytes = wc::repair_unit_bytes(a.group, a.head_dim, max_repair_blocks, r.tiles);
  return hip_status(wc::launch_repair(r, static_cast<hipStream_t>(stream)));
}

size_t wc_block_repair_workspace_size(int batch, int n_q_heads, int n_kv_heads, int head_dim,
                                      int max_repair_blocks) {
  if (batch < 0 || n_kv_heads < 1 || n_q_heads < 1 || n_q_heads % n_kv_heads || head_dim < 1 ||
      max_repair_blocks < 1 || max_repair_blocks > 64)
    return 0;
  const size_t unit = wc::repair_unit_bytes(n_q_heads / n_kv_heads, head_dim, max_repair_blocks,
                                            wc::kRepairTiles);
  const size_t total = (size_t)batch * n_kv_heads * unit;
  return total > 0 ? total : 256;
}

int wc_repair_write_back(const wc_cache* cache, int batch, const int32_t* block_table,
                         int max_blocks_per_seq, const int32_t* seq_lens, const int32_t* repaired_blocks,
                         const int32_t* n_repaired, int max_repair_blocks, const uint8_t* whole_kv,
                         void* stream) {
  if (cache == nullptr || cache->repaired == nullptr) return WC_EINVAL;
  const int s = check_cache(cache, false, true);
  if (s != WC_OK) return s;
  if (batch < 0 || max_blocks_per_seq < 1) return WC_EINVAL;
  if (n_repaired != nullptr && (max_repair_blocks < 1 || max_repair_blocks > 64 || !repaired_blocks))
    return WC_EINVAL;
  if (batch == 0 || (n_repaired == nullptr && whole_kv == nullptr)) return WC_OK;
  if (!block_table || !seq_lens) return WC_EINVAL;
  wc::WriteBackArgs w{};
  w.repaired = cache->repaired;
  w.k_witness = static_cast<uint16_t*>(cache->k_witness);
  w.num_blocks = cache->num_blocks;
  w.n_kv = cache->n_kv_heads;
  w.n_bands = cache->n_bands;
  w.batch = batch;
  w.max_blocks = max_blocks_per_seq;
  w.max_rep = n_repaired != nullptr ? max_repair_blocks : 1;
  w.table = block_table;
  w.seq_lens = seq_lens;
  w.list = repaired_blocks;
  w.n_rep = n_repaired;
  w.whole_kv = whole_kv;
  return hip_status(wc::launch_write_back(w, static_cast<hipStream_t>(stream)));
}

int wc_gate(const float* meter, const float* raw, int batch, int n_q_heads, int group, float tau,
            uint8_t* mask_q, uint8_t* mask_kv, int32_t* n_gated, void* stream) {
  if (batch < 0 || n_q_heads < 1 || group < 1 || n_q_heads % group || !(tau >= 0.0f)) return WC_EINVAL;
  if (batch == 0) return WC_OK;
  if (!mask_q || !mask_kv || (tau < 1.0f ? !meter : !raw)) return WC_EINVAL;
  wc::GateArgs a{meter, raw, mask_q, mask_kv, n_gated, batch, n_q_heads, group, tau};
  return hip_status(wc::launch_gate(a, static_cast<hipStream_t>(stream)));
}

int wc_exact_decode_attention(const wc_cache* exact, const void* q, int q_dtype, int batch,
                              int n_q_heads, const int32_t* block_table,
                              int max_blocks_per_seq, const int32_t* seq_lens,
                              int64_t max_seq_len, float sm_scale, const uint8_t* mask_kv,
                              void* out, int out_dtype, int split_tokens, void* ws,
                              size_t ws_bytes, void* stream) {
  int s = check_cache(exact, false);
  if (s != WC_OK) return s;
  if (exact->kind != WC_KIND_BF16) return WC_EINVAL;
  if (batch > 0 && !mask_kv) return WC_EINVAL;
  wc::DecodeArgs a{};
  s = decode_common(exact, q, q_dtype, batch, n_q_heads, block_table, max_blocks_per_seq,
                    seq_lens, max_seq_len, sm_scale, out, out_dtype, split_tokens, ws, ws_bytes, a);
  if (s != WC_OK) return s;
  a.mask_kv = mask_kv;
  a.meter = nullptr;
  a.raw = nullptr;
  return hip_status(wc::launch_decode(a, false, static_cast<hipStream_t>(stream)));
}

}  // extern "C"
