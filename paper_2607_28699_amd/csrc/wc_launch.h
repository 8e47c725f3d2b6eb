// Kernel argument blocks and launchers behind the C-ABI (host + device visible).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/witcert.h"
#include "wc_device.h"

namespace wc {

struct WriteArgs {
  int kind, head_dim, n_kv, n_bands, interleaved, layer, in_dtype;
  uint32_t key0, key1;
  int64_t n_tok;
  int64_t n_slots;          // slots of the cache(s): a slot outside [0, n_slots) is skipped
  const void* k;
  const void* v;
  const int64_t* slots;
  void* k_data;
  void* v_data;
  uint16_t* k_scale;
  uint16_t* v_scale;
  uint16_t* k_witness;
  void* x_k_data;           // bf16 exact cache written in the same pass (or null)
  void* x_v_data;
  int n_pairs;              // bypassed RoPE pairs per KV head (0: none)
  const int32_t* pairs;     // [n_kv][n_pairs]
  uint16_t* k_outlier;      // [blocks][n_kv][16][2 n_pairs] fp16
  uint16_t* v_resid;        // value side (or null): ||vhat - v|| fp16 up, [blocks][n_kv][16]
  uint16_t* v_norm;         // ||v|| fp16 down, same layout
  int group_scales;         // k_scale / v_scale hold one fp16 scale per 32-channel group
};

struct SelectArgs {
  const void* k;
  int in_dtype, n_kv, head_dim, interleaved, m, n_chunks;
  int64_t n_tok;
  int32_t* pairs_out;
  double* part;             // [n_kv][n_chunks][head_dim / 2] partial pair energies (workspace)
};

struct WitnessArgs {
  const void* x;
  const void* xhat;
  int x_dtype, xhat_dtype, head_dim, n_bands, interleaved;
  int64_t n_vec;
  uint16_t* w_out;
};

// Decode: one split (a contiguous chunk of split_tokens tokens) of one
// (sequence, KV head) per workgroup; partial records merged by a second kernel.
struct DecodeArgs {
  const void* k_data;
  const void* v_data;
  const uint16_t* k_scale;
  const uint16_t* v_scale;
  const uint16_t* k_witness;
  const void* q;
  const int32_t* table;
  const int32_t* seq_lens;
  int64_t num_blocks;       // blocks of the cache(s) read: a table entry outside [0, num_blocks)
                            // is read as a page of zeros (no access outside the cache)
  const uint8_t* mask_kv;   // exact fallback: only routed (b, kv) units run
  float* part;              // partial records [batch][n_q][n_splits][D + 8]
  // meter numerators of block segments (metered decodes; null: not recorded):
  // [batch][n_q][n_splits][share_slots] float4 (see share_slots())
  float4* shares;
  int share_slots;
  void* out;
  float* meter;
  float* raw;
  int kind, head_dim, n_bands, interleaved, q_dtype, out_dtype;
  int batch, n_q, n_kv, group, max_blocks, n_splits, split_tokens, layer;
  uint32_t key0, key1;
  float sm_scale;
  int use_mfma;             // matrix-core kernels where supported (else the vector path)
  float tierb_delta;        // > 0: Tier-B radius (u_t = (alpha_h + beta_h) s_t) instead of the witness
  // gate applied in the split merge (null gate_mask_q: no gate)
  uint8_t* gate_mask_q;     // [batch][n_q]
  uint8_t* gate_mask_kv;    // [batch][n_kv], cleared by the decode kernel
  int32_t* gate_unit;       // [batch][n_kv] gated-head counts (workspace), cleared likewise
  int32_t* gate_count;      // device int32[2] or null
  float gate_tau;
  int n_pairs;              // bypassed RoPE pairs per KV head (0: none)
  const int32_t* pairs;     // [n_kv][n_pairs]
  const uint16_t* k_outlier;  // [blocks][n_kv][16][2 n_pairs] fp16
  // value side (null meter_v: off): stored ||vhat - v|| (up) and ||v|| (down), the
  // value meter out, and its threshold in the joint gate
  const uint16_t* v_resid;
  const uint16_t* v_norm;
  float* meter_v;           // [batch][n_q]
  float gate_tau_v;
  // k_scale / v_scale hold one fp16 scale per 32-channel group ([..][16][D/32]),
  // else one per token
  int group_scales;
  // a decode step's new tokens (one per sequence, its last): written by the
  // matrix-core decode before it reads them (step_write != 0), else nothing
  WriteArgs sw;
  int step_write;
  // persistent repair: pages marked in repaired[blk * n_kv + kv] are read from the
  // exact store (bf16 pages x_k_data / x_v_data) with bound 0 (null: no marks)
  const uint8_t* repaired;
  const void* x_k_data;
  const void* x_v_data;
  // certified step (metered decode, exact fallback, final merge): the exact
  // fallback decides each unit's gate from the metered records gate_part (same
  // split layout) in its prologue; the final merge takes routed heads' outputs
  // from the exact records x_part (null: not in use)
  const float* gate_part;
  const float* x_part;
  int no_merge;             // launch_decode: the decode kernel only (the merge comes later)
  // speculative certified step: the exact records x_part cover every unit, and the
  // final merge decides each unit's gate itself from the metered records (gate_part)
  int merge_gate;
};

// Scale of channel c of the token in scale row `row` (page * 16 + offset): the
// token's, or with group scales that of its 32-channel group.
__device__ __forceinline__ float scale_of(const uint16_t* sc, int64_t row, int c, int D, bool grouped) {
  return f16_to_f32(grouped ? sc[row * (D / 32) + (c >> 5)] : sc[row]);
}

// Channel of member `second` of RoPE pair j (pair index clamped into range).
__host__ __device__ inline int pair_channel(int j, int second, int d, bool interleaved) {
  j = j < 0 ? 0 : (j >= d / 2 ? d / 2 - 1 : j);
  return interleaved ? 2 * j + second : j + second * (d / 2);
}

// Tier-B factor (alpha + beta) of one query head: u_t = (alpha + beta) * s_t with
// alpha = sm ||q|| sqrt(2 log(2S / delta) / 12) (Sec. 4.2, Tier B; the square root
// hoisted out of the token loop, Sec. 6.2 serving integration) and beta =
// sm ||q||_1 / 256, the mean of the 8-bit dither lattice's residual.
__device__ __forceinline__ float tierb_factor(float q_sq, float q_l1, int n_tokens, float delta,
                                             float sm_scale) {
  const float lg = logf(2.0f * (float)n_tokens / delta);
  return sm_scale * (sqrtf(q_sq) * sqrtf(2.0f * lg / 12.0f) + q_l1 * (1.0f / 256.0f));
}

// Decode grids hold n_splits x (batch x n_kv) workgroups, one per (sequence, KV
// head, split).  Workgroups go to the eight XCDs round-robin in linear order, and
// the KV heads of one block read the same 128-byte lines of the per-token arrays
// (scales, value side: [block][kv][16] fp16, 32 bytes per KV head), so the linear
// order puts the n_kv heads of one (sequence, split) 8 apart -- on one XCD, where
// its L2 serves the line to all of them.  Positions P = (sequence, split) go in
// groups of 8 (one per XCD; a last partial group fills the rest), and each
// sequence's splits are rotated by the sequence index, so that the sequences'
// first splits -- always present, while later ones exist only for long sequences
// -- spread over the XCDs too.
struct DecodePos {
  int unit;    // sequence x n_kv + KV head
  int split;
};
__device__ __forceinline__ DecodePos decode_position_at(uint32_t L, int batch, int n_kv, int n_splits) {
  const uint32_t K = (uint32_t)n_kv, NS = (uint32_t)n_splits;
  const uint32_t nP = (uint32_t)batch * NS;
  const uint32_t full = nP / 8u * 8u;   // positions in whole groups of 8
  uint32_t P, kv;
  if (L < full * K) {
    const uint32_t grp = L / (8u * K), rem = L % (8u * K);
    kv = rem / 8u;
    P = 8u * grp + rem % 8u;
  } else {
    const uint32_t Lr = L - full * K, R = nP - full;
    kv = Lr / R;
    P = full + Lr % R;
  }
  const uint32_t b = P / NS, s = P % NS;
  return DecodePos{(int)(b * K + kv), (int)((s + b) % NS)};
}
__device__ __forceinline__ DecodePos decode_position(int batch, int n_kv, int n_splits) {
  return decode_position_at(blockIdx.x + gridDim.x * blockIdx.y, batch, n_kv, n_splits);
}

// Clears the gate outputs of one (sequence, KV head) ahead of the merge.
__device__ __forceinline__ void gate_clear(const DecodeArgs& a, int unit, int split) {
  if (a.gate_mask_q != nullptr && a.gate_part == nullptr && split == 0 && threadIdx.x == 0) {
    a.gate_mask_kv[unit] = 0;
    a.gate_unit[unit] = 0;
  }
}

// Block repair (Sec. 6.3): the decode arguments of the call that routed the KV
// heads (its records in d.part, d.mask_kv the routed units), the exact cache, the
// threshold and the repair budget.
struct RepairArgs {
  DecodeArgs d;
  const void* x_k_data;     // exact bf16 cache
  const void* x_v_data;
  float tau;
  int max_rep;              // blocks per KV head, <= 64
  uint8_t* mask_kv_out;     // cleared for repaired KV heads (the same array as d.mask_kv)
  int32_t* rep_list;        // [batch][n_kv][max_rep] block order (-1 padded), or null
  int32_t* n_rep;           // [batch][n_kv] blocks taken, 0 not routed, -1 not repaired; or null
  void* rws;                // repair workspace: per (sequence, KV head) a header and the
                            // corrections of every (candidate block, 64-token tile)
  size_t unit_bytes;        // workspace bytes per (sequence, KV head)
  int tiles;                // 64-token tiles per block
  int round0_cap;           // > 0: blocks in the first correction round (else the predicted count + 1)
};
constexpr int kRepHeaderBytes = 1024;

// Write-back of a repair (persistent repair): marks and zeroed witnesses.
struct WriteBackArgs {
  uint8_t* repaired;        // [num_blocks][n_kv]
  uint16_t* k_witness;      // [num_blocks][n_kv][16][n_bands] or null
  int64_t num_blocks;
  int n_kv, n_bands, batch, max_blocks, max_rep;
  const int32_t* table;
  const int32_t* seq_lens;
  const int32_t* list;      // [batch][n_kv][max_rep] repaired blocks
  const int32_t* n_rep;     // [batch][n_kv] or null
  const uint8_t* whole_kv;  // [batch][n_kv] or null
};
hipError_t launch_write_back(const WriteBackArgs& w, hipStream_t st);
// Repair blocks: fixed runs of 256 tokens of the sequence (Sec. 6.3), corrected in
// 64-token tiles.
constexpr int kRepairBlockTokens = 256;
constexpr int kRepairTiles = kRepairBlockTokens / 64;
// Repair workspace bytes per (sequence, KV head) (a multiple of 256).
size_t repair_unit_bytes(int group, int head_dim, int max_rep, int tiles);

struct GateArgs {
  const float* meter;
  const float* raw;
  uint8_t* mask_q;
  uint8_t* mask_kv;
  int32_t* n_gated;
  int batch, n_q, group;
  float tau;
};

// Tokens per KV split chosen by the library (multiple of 64): about `target`
// (sequence, KV head, split) workgroups -- 512, two per compute unit, for the decode
// calls; 256 for the speculative certified step, whose one launch holds twice the
// workgroups of a decode.
constexpr int64_t kDecodeWorkgroups = 512;
int choose_split_tokens(int batch, int n_kv, int64_t max_seq_len, int requested,
                        int64_t target = kDecodeWorkgroups);
// The same, balanced over the batch's total tokens (ragged batches).
int choose_split_tokens_total(int n_kv, int64_t max_seq_len, int64_t total_tokens,
                              int64_t target = kDecodeWorkgroups);
inline int64_t n_splits_for(int64_t max_seq_len, int split_tokens) {
  return max_seq_len <= 0 ? 1 : (max_seq_len + split_tokens - 1) / split_tokens;
}
// Partial record of one (query head, split): head_dim output floats, then the
// running max (natural log units), weight sum, meter numerator, value-side
// numerator sum p rho, the largest stored value norm and three spare floats.
// Weights are e^{logit - max}; the record is a multiple of 16 bytes.
__host__ __device__ inline size_t partial_record_floats(int head_dim) { return (size_t)head_dim + 8; }
// Block segments of a metered decode (block repair's shares, Sec. 6.3): a segment
// is the part of one work item's token range (a matrix-core wave's pages, the
// vector path's split) that lies in one 256-token repair block.  Each (query head,
// split) has share_slots() entries float4 {numerator sum_t e^{logit_t - m}
// (e^{c_t} - 1) over the segment, frame m (natural log), first page (int bits),
// pages (int bits, 0: unused slot)}; the matrix-core wave w owns slots
// [w * S / 4, (w + 1) * S / 4), the vector path's workgroup all S of its split, and
// every owned slot is written.
inline int share_slots(int split_tokens) {
  const int pages = split_tokens / 16;
  const int ppw = (pages + 3) / 4;                        // pages of one wave, at most
  const int per_wave = (ppw + 14) / 16 + 1;              // repair blocks such a run can touch
  const int per_split = (pages + 14) / 16 + 1;
  const int q = per_wave > (per_split + 3) / 4 ? per_wave : (per_split + 3) / 4;
  return 4 * q;
}
// Workspace: the partial records, one int32 per (sequence, KV head) for the fused
// gate, then the block segments; each part rounded up to 256 bytes.
inline size_t records_bytes(int batch, int n_q, int64_t n_splits, int head_dim) {
  const size_t b = (size_t)batch * n_q * n_splits * partial_record_floats(head_dim) * sizeof(float);
  return (b + 255) / 256 * 256;
}
inline size_t gate_unit_bytes(int batch, int n_kv) {
  return ((size_t)batch * n_kv * sizeof(int32_t) + 255) / 256 * 256;
}
inline size_t share_bytes(int batch, int n_q, int64_t n_splits, int split_tokens) {
  return (size_t)batch * n_q * n_splits * share_slots(split_tokens) * 16;
}

hipError_t launch_quantize_write(const WriteArgs& a, hipStream_t st);
hipError_t launch_witness(const WitnessArgs& a, hipStream_t st);
hipError_t launch_select_pairs(const SelectArgs& a, hipStream_t st);
int select_chunks(int64_t n_tok);   // row chunks of the pair-energy pass
hipError_t launch_decode(const DecodeArgs& a, bool metered, hipStream_t st);
bool mfma_decode_supported(const DecodeArgs& a);
hipError_t launch_decode_mfma(const DecodeArgs& a, bool metered, hipStream_t st);
// The decode call would run on the matrix cores (where a step's new tokens can be
// written by the decode kernel itself).
bool step_write_fusable(const DecodeArgs& a);
// The speculative certified step's metered decode (am, plain Tier A) and exact
// fallback of every unit (ax) can share one matrix-core launch.
bool spec_decode_fusable(const DecodeArgs& am, const DecodeArgs& ax);
hipError_t launch_decode_spec(const DecodeArgs& am, const DecodeArgs& ax, hipStream_t st);
hipError_t launch_merge(const DecodeArgs& a, bool metered, hipStream_t st);
hipError_t launch_gate(const GateArgs& a, hipStream_t st);
hipError_t launch_repair(const RepairArgs& a, hipStream_t st);
int repair_max_blocks();

}  // namespace wc
