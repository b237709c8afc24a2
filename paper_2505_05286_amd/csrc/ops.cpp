// C ABI of the individual kernels (include/hxf_ops.h).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <vector>

#include "decode_plan.hpp"
#include "executor.hpp"
#include "hxf_ops.h"
#include "kernels/kernels.hpp"

using namespace hxf;

namespace {

int64_t al(int64_t x) { return (x + 255) & ~int64_t(255); }

int dev_rc(hipError_t e) { return e == hipSuccess ? HXF_OK : HXF_EDEVICE; }

struct DecodeLayout {
  int64_t items = 0, merges = 0, parts = 0, off_items = 0, off_merges = 0, off_qrow = 0, off_o = 0, off_ml = 0,
          total = 0;
};

void decode_seqs(int B, const int32_t* ctx, const int32_t* bt_host, int bt_stride, std::vector<DecodeSeq>& seqs) {
  seqs.clear();
  for (int b = 0; b < B; ++b)
    seqs.push_back(DecodeSeq{b, std::max(ctx[b], 1), bt_host ? bt_host + (size_t)b * bt_stride : nullptr});
}

DecodeLayout decode_layout(const DecodePlan& P, int B, int Hq, int Hkv, int dh) {
  DecodeLayout L;
  L.items = (int64_t)P.items.size();
  L.merges = (int64_t)B * Hkv;
  L.parts = P.n_parts;
  const int G = Hq / Hkv;
  int64_t o = 0;
  L.off_items = o; o = al(o + L.items * (int64_t)sizeof(DecodeItem));
  L.off_merges = o; o = al(o + L.merges * (int64_t)sizeof(MergeItem));
  L.off_qrow = o; o = al(o + (int64_t)B * 4);
  L.off_o = o; o = al(o + L.parts * G * dh * 4);
  L.off_ml = o; o = al(o + L.parts * G * 2 * 4);
  L.total = o;
  return L;
}

bool shapes_ok(int Hq, int Hkv, int dh) {
  return Hq > 0 && Hkv > 0 && Hq % Hkv == 0 && Hq / Hkv <= 16 && (dh == 64 || dh == 128);
}

// memcpy of a vector's elements; nothing for an empty one (whose data() may be null)
template <typename T>
void copy_vec(void* dst, const std::vector<T>& v) {
  if (!v.empty()) std::memcpy(dst, v.data(), v.size() * sizeof(T));
}

}  // namespace

extern "C" {

int64_t hxf_op_gemm_workspace_bytes(int32_t M, int32_t N, int32_t K) {
  if (M <= 0 || N <= 0 || K <= 0) return 0;
  // enough for every epilogue (the SwiGLU plan may differ)
  int64_t need = 0;
  for (bool sw : {false, true}) {
    const GemmPlan p = gemm_plan(M, N, K, 8, sw);
    if (p.splits > 1) need = std::max(need, (int64_t)p.splits * M * N * 4);
  }
  return need;
}

int hxf_op_gemm(const void* A, int32_t lda, const void* B, const void* B2, void* C, int32_t ldc, int32_t M, int32_t N,
                int32_t K, int32_t flags, void* workspace, int64_t ws_bytes, void* stream) {
  const int epi = flags & 0xFF;
  const bool a_packed = flags & HXF_GEMM_A_PACKED, c_packed = flags & HXF_GEMM_C_PACKED;
  if (flags & ~(0xFF | HXF_GEMM_A_PACKED | HXF_GEMM_C_PACKED)) return HXF_EINVAL;
  if (!A || !B || !C || M < 0 || N <= 0 || K <= 0 || K % 8 || (!a_packed && lda < K) || epi < 0 || epi > 3)
    return HXF_EINVAL;
  if (epi == HXF_EPI_SWIGLU && (!B2 || N % 32)) return HXF_EINVAL;
  if (!c_packed && ldc < (epi == HXF_EPI_SWIGLU ? N / 2 : N)) return HXF_EINVAL;
  if ((a_packed && (K % 32 || (epi == HXF_EPI_SWIGLU && N % 64))) || (c_packed && (epi != HXF_EPI_SWIGLU || N % 64)))
    return HXF_EINVAL;
  if (M == 0) return HXF_OK;
  GemmPlan p = gemm_plan(M, N, K, 8, epi == HXF_EPI_SWIGLU);
  if (p.splits > 1 && (!workspace || ws_bytes < (int64_t)p.splits * M * N * 4)) return HXF_ENOMEM;
  GemmArgs a{};
  a.A = (const uint16_t*)A;
  a.B = (const uint16_t*)B;
  a.B2 = (const uint16_t*)B2;
  a.C = C;
  a.partial = (float*)workspace;
  a.M = M;
  a.N = N;
  a.K = K;
  a.lda = lda;
  a.ldc = ldc;
  a.kt = (K + 31) / 32;
  a.a_packed = a_packed ? 1 : 0;
  a.c_kt = c_packed ? N / 64 : 0;
  return dev_rc(gemm_launch(a, epi, p, (hipStream_t)stream));
}

int64_t hxf_packed_weight_bytes(int32_t N, int32_t K) {
  if (N <= 0 || K <= 0) return 0;
  return (int64_t)packed_weight_elems(N, K) * 2;
}

int hxf_op_pack_weight(const void* W, int32_t N, int32_t K, void* out, void* stream) {
  if (!W || !out || N <= 0 || K <= 0 || K % 8) return HXF_EINVAL;
  return dev_rc(pack_weight_launch((const uint16_t*)W, N, K, (uint16_t*)out, (hipStream_t)stream));
}

int hxf_op_rmsnorm(const float* x, const int32_t* rows, const void* g, void* out, int32_t n_rows, int32_t d, float eps,
                   void* stream) {
  if (!x || !g || !out || n_rows < 0 || d <= 0 || d % 4) return HXF_EINVAL;
  return dev_rc(rmsnorm_launch(x, rows, (const uint16_t*)g, (uint16_t*)out, n_rows, d, eps, (hipStream_t)stream));
}

int hxf_op_embed_rmsnorm(const int32_t* ids, const void* E, const void* g, float* resid, void* out, int32_t T,
                         int32_t d, float eps, void* stream) {
  if (!ids || !E || !g || !resid || !out || T < 0 || d <= 0 || d % 4) return HXF_EINVAL;
  return dev_rc(embed_rmsnorm_launch(ids, (const uint16_t*)E, (const uint16_t*)g, resid, (uint16_t*)out, T, d, eps,
                                     (hipStream_t)stream));
}

int hxf_op_rope_table(void* dst, int32_t max_pos, int32_t dh, float base, void* stream) {
  if (!dst || max_pos <= 0 || dh <= 0 || dh % 2) return HXF_EINVAL;
  std::vector<float> t;
  build_rope_table(t, max_pos, dh, base);
  hipStream_t st = (hipStream_t)stream;
  if (hipMemcpyAsync(dst, t.data(), t.size() * 4, hipMemcpyHostToDevice, st) != hipSuccess) return HXF_EDEVICE;
  return dev_rc(hipStreamSynchronize(st));
}

int hxf_op_rope_kv_write(void* qkv, const int32_t* pos, const int32_t* slot, const void* table, void* k_pool,
                         void* v_pool, int64_t n_blocks, int32_t T, int32_t Hq, int32_t Hkv, int32_t dh, void* stream) {
  if (!qkv || !pos || !slot || !table || !k_pool || !v_pool || n_blocks <= 0 || T < 0 || !shapes_ok(Hq, Hkv, dh))
    return HXF_EINVAL;
  return dev_rc(rope_kv_launch((uint16_t*)qkv, pos, slot, (const float2*)table, (uint16_t*)k_pool,
                               (uint16_t*)v_pool, n_blocks, T, Hq, Hkv, dh, (hipStream_t)stream));
}

int hxf_op_kv_scatter(const void* k, const void* v, const int32_t* slot, void* k_pool, void* v_pool, int64_t n_blocks,
                      int32_t T, int32_t Hkv, int32_t dh, void* stream) {
  if (!k || !v || !slot || !k_pool || !v_pool || n_blocks <= 0 || T < 0 || Hkv <= 0 || dh <= 0) return HXF_EINVAL;
  return dev_rc(kv_scatter_launch((const uint16_t*)k, (const uint16_t*)v, slot, (uint16_t*)k_pool,
                                  (uint16_t*)v_pool, n_blocks, T, Hkv, dh, (hipStream_t)stream));
}

int64_t hxf_op_decode_attention_workspace_bytes(int32_t B, int32_t Hq, int32_t Hkv, int32_t dh, const int32_t* ctx,
                                                const int32_t* bt_host, int32_t bt_stride) {
  if (B < 0 || !ctx || !shapes_ok(Hq, Hkv, dh) || (bt_host && bt_stride <= 0)) return -1;
  std::vector<DecodeSeq> seqs;
  decode_seqs(B, ctx, bt_host, bt_stride, seqs);
  DecodePlan P;
  plan_decode(seqs, Hkv, Hq / Hkv, P);
  return decode_layout(P, B, Hq, Hkv, dh).total;
}

int hxf_op_decode_plan(int32_t B, int32_t Hq, int32_t Hkv, const int32_t* ctx, const int32_t* bt_host, int32_t bt_stride,
                       int32_t* items, int32_t items_cap, int32_t* n_items, int32_t* merges, int32_t merges_cap,
                       int32_t* n_merges) {
  if (B < 0 || !ctx || Hq <= 0 || Hkv <= 0 || Hq % Hkv || Hq / Hkv > 16 || (bt_host && bt_stride <= 0) || !n_items ||
      !n_merges || (items_cap > 0 && !items) || (merges_cap > 0 && !merges))
    return HXF_EINVAL;
  std::vector<DecodeSeq> seqs;
  decode_seqs(B, ctx, bt_host, bt_stride, seqs);
  DecodePlan P;
  plan_decode(seqs, Hkv, Hq / Hkv, P);
  *n_items = (int32_t)P.items.size();
  *n_merges = (int32_t)P.merges.size();
  if ((int64_t)items_cap < (int64_t)P.items.size() || (int64_t)merges_cap < (int64_t)P.merges.size())
    return HXF_ENOMEM;
  copy_vec(items, P.items);
  copy_vec(merges, P.merges);
  return HXF_OK;
}

int hxf_op_decode_attention(const void* q, const void* k_pool, const void* v_pool, int64_t n_blocks, const int32_t* bt,
                            int32_t bt_stride, const int32_t* ctx, const int32_t* bt_host, void* out, int32_t B,
                            int32_t Hq, int32_t Hkv, int32_t dh, void* workspace, int64_t ws_bytes, void* stream) {
  if (!q || !k_pool || !v_pool || n_blocks <= 0 || !bt || !ctx || !out || B < 0 || !shapes_ok(Hq, Hkv, dh))
    return HXF_EINVAL;
  if (B == 0) return HXF_OK;
  for (int b = 0; b < B; ++b)
    if (ctx[b] <= 0 || (ctx[b] + kPage - 1) / kPage > bt_stride) return HXF_EINVAL;
  std::vector<DecodeSeq> seqs;
  decode_seqs(B, ctx, bt_host, bt_stride, seqs);
  DecodePlan P;
  plan_decode(seqs, Hkv, Hq / Hkv, P);
  const DecodeLayout L = decode_layout(P, B, Hq, Hkv, dh);
  if (!workspace || ws_bytes < L.total) return HXF_ENOMEM;
  std::vector<uint8_t> host(L.off_o);
  copy_vec(host.data() + L.off_items, P.items);
  copy_vec(host.data() + L.off_merges, P.merges);
  auto* qrow = reinterpret_cast<int32_t*>(host.data() + L.off_qrow);
  for (int b = 0; b < B; ++b) qrow[b] = b;
  hipStream_t st = (hipStream_t)stream;
  uint8_t* ws = (uint8_t*)workspace;
  if (hipMemcpyAsync(ws, host.data(), host.size(), hipMemcpyHostToDevice, st) != hipSuccess) return HXF_EDEVICE;
  DecodeAttnArgs a{};
  a.q = (const uint16_t*)q;
  a.q_row = reinterpret_cast<const int32_t*>(ws + L.off_qrow);
  a.q_stride = Hq * dh;
  a.k_pool = (const uint16_t*)k_pool;
  a.v_pool = (const uint16_t*)v_pool;
  a.n_blocks = n_blocks;
  a.bt = bt;
  a.bt_stride = bt_stride;
  a.items = reinterpret_cast<const DecodeItem*>(ws + L.off_items);
  a.n_items = (int)(P.items.size() - P.n_wide);
  a.n_wide = (int)P.n_wide;
  a.merges = reinterpret_cast<const MergeItem*>(ws + L.off_merges);
  a.n_merges = (int)L.merges;
  a.part_o = reinterpret_cast<float*>(ws + L.off_o);
  a.part_ml = reinterpret_cast<float*>(ws + L.off_ml);
  a.out = (uint16_t*)out;
  a.out_stride = Hq * dh;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.dh = dh;
  a.scale_log2 = 1.4426950408889634f / std::sqrt((float)dh);
  if (decode_attn_launch(a, st) != hipSuccess || decode_merge_launch(a, st) != hipSuccess) return HXF_EDEVICE;
  return dev_rc(hipStreamSynchronize(st));
}

namespace {

// Workspace of hxf_op_prefill_attention: items (whole ones plus the parts of split
// ones), merge jobs, row0 / pos0, then the partial outputs and (max, sum) of the parts.
struct PrefillLayout {
  int64_t off_merges = 0, off_rp = 0, off_o = 0, off_ml = 0, total = 0;
};

PrefillLayout prefill_layout(int64_t whole_items, int S, int dh) {
  PrefillLayout L;
  const int64_t items = whole_items + kPrefillResident, parts = prefill_parts_bound(whole_items);
  int64_t o = al(items * (int64_t)sizeof(PrefillItem));
  L.off_merges = o;
  o = al(o + whole_items * (int64_t)sizeof(PrefillMerge));
  L.off_rp = o;
  o = al(o + (int64_t)S * 8);
  L.off_o = o;
  o = al(o + parts * kPrefillPairs * dh * 4);
  L.off_ml = o;
  L.total = al(o + parts * kPrefillPairs * 2 * 4);
  return L;
}

int64_t prefill_whole_items(int S, int Hkv, int qpi, const int32_t* n_host) {
  int64_t items = 0;
  for (int s = 0; s < S; ++s) items += (int64_t)Hkv * ((n_host[s] + qpi - 1) / qpi);
  return items;
}

}  // namespace

int64_t hxf_op_prefill_attention_workspace_bytes(int32_t S, int32_t Hq, int32_t Hkv, const int32_t* n_host) {
  if (S < 0 || !n_host || Hq <= 0 || Hkv <= 0 || Hq % Hkv) return -1;
  const int qpi = prefill_queries_per_item(Hq / Hkv);
  // head_dim is not an argument: size the partials for the largest (128)
  return prefill_layout(prefill_whole_items(S, Hkv, qpi, n_host), S, 128).total;
}

int hxf_op_prefill_plan(int32_t S, int32_t Hq, int32_t Hkv, const int32_t* pos0, const int32_t* n_host,
                        int32_t* items, int32_t items_cap, int32_t* n_items, int32_t* merges, int32_t merges_cap,
                        int32_t* n_merges) {
  if (S < 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv || Hq / Hkv > 16 || (S > 0 && (!pos0 || !n_host)) || !n_items ||
      !n_merges || (items_cap > 0 && !items) || (merges_cap > 0 && !merges))
    return HXF_EINVAL;
  std::vector<PrefillEntry> entries;
  for (int s = 0; s < S; ++s) {
    if (n_host[s] < 0 || pos0[s] < 0) return HXF_EINVAL;
    if (n_host[s] > 0) entries.push_back(PrefillEntry{s, pos0[s], n_host[s]});
  }
  PrefillPlan P;
  plan_prefill(entries, Hkv, prefill_queries_per_item(Hq / Hkv), P);
  *n_items = (int32_t)P.items.size();
  *n_merges = (int32_t)P.merges.size();
  if ((int64_t)items_cap < (int64_t)P.items.size() || (int64_t)merges_cap < (int64_t)P.merges.size())
    return HXF_ENOMEM;
  copy_vec(items, P.items);
  copy_vec(merges, P.merges);
  return HXF_OK;
}

int hxf_op_prefill_attention(const void* q, const void* k_pool, const void* v_pool, int64_t n_blocks, const int32_t* bt,
                             int32_t bt_stride, const int32_t* row0, const int32_t* pos0, const int32_t* n_host,
                             void* out, int32_t S, int32_t Hq, int32_t Hkv, int32_t dh, void* workspace,
                             int64_t ws_bytes, void* stream) {
  if (!q || !k_pool || !v_pool || n_blocks <= 0 || !bt || !row0 || !pos0 || !n_host || !out || S < 0 ||
      !shapes_ok(Hq, Hkv, dh))
    return HXF_EINVAL;
  if (S == 0) return HXF_OK;
  for (int s = 0; s < S; ++s)
    if (n_host[s] < 0 || pos0[s] < 0 || row0[s] < 0 || (pos0[s] + n_host[s] + kPage - 1) / kPage > bt_stride)
      return HXF_EINVAL;
  const int64_t need = hxf_op_prefill_attention_workspace_bytes(S, Hq, Hkv, n_host);
  if (!workspace || ws_bytes < need) return HXF_ENOMEM;
  const int qpi = prefill_queries_per_item(Hq / Hkv);
  std::vector<PrefillEntry> entries;
  for (int s = 0; s < S; ++s)
    if (n_host[s] > 0) entries.push_back(PrefillEntry{s, pos0[s], n_host[s]});
  PrefillPlan P;
  plan_prefill(entries, Hkv, qpi, P);
  const PrefillLayout L = prefill_layout(prefill_whole_items(S, Hkv, qpi, n_host), S, 128);
  std::vector<uint8_t> host(L.off_rp + (int64_t)S * 8);
  copy_vec(host.data(), P.items);
  copy_vec(host.data() + L.off_merges, P.merges);
  std::memcpy(host.data() + L.off_rp, row0, (size_t)S * 4);
  std::memcpy(host.data() + L.off_rp + S * 4, pos0, (size_t)S * 4);
  hipStream_t st = (hipStream_t)stream;
  uint8_t* ws = (uint8_t*)workspace;
  if (hipMemcpyAsync(ws, host.data(), host.size(), hipMemcpyHostToDevice, st) != hipSuccess) return HXF_EDEVICE;
  PrefillAttnArgs a{};
  a.q = (const uint16_t*)q;
  a.q_stride = Hq * dh;
  a.row0 = reinterpret_cast<const int32_t*>(ws + L.off_rp);
  a.pos0 = reinterpret_cast<const int32_t*>(ws + L.off_rp + S * 4);
  a.k_pool = (const uint16_t*)k_pool;
  a.v_pool = (const uint16_t*)v_pool;
  a.n_blocks = n_blocks;
  a.bt = bt;
  a.bt_stride = bt_stride;
  a.items = reinterpret_cast<const PrefillItem*>(ws);
  a.n_items = (int)P.items.size();
  a.merges = reinterpret_cast<const PrefillMerge*>(ws + L.off_merges);
  a.n_merges = (int)P.merges.size();
  a.part_o = reinterpret_cast<float*>(ws + L.off_o);
  a.part_ml = reinterpret_cast<float*>(ws + L.off_ml);
  a.out = (uint16_t*)out;
  a.out_stride = Hq * dh;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.dh = dh;
  a.scale_log2 = 1.4426950408889634f / std::sqrt((float)dh);
  if (prefill_attn_launch(a, st) != hipSuccess) return HXF_EDEVICE;
  return dev_rc(hipStreamSynchronize(st));
}

int hxf_op_argmax(const float* logits, int32_t* out, int32_t R, int32_t V, void* stream) {
  if (!logits || !out || R < 0 || V <= 0 || V % 4) return HXF_EINVAL;
  return dev_rc(argmax_launch(logits, out, R, V, (hipStream_t)stream));
}

int hxf_op_copy(const void* src, void* dst, int64_t bytes, void* stream) {
  if (!src || !dst || bytes < 0 || bytes % 16) return HXF_EINVAL;
  return dev_rc(copy_launch(src, dst, (size_t)bytes, (hipStream_t)stream));
}

int hxf_op_read(const void* src, int64_t bytes, uint32_t* sink, void* stream) {
  static_assert(HXF_READ_SINK_WORDS == kReadProbeBlocks * 256, "sink size");
  if (!src || !sink || bytes < 0 || bytes % 16) return HXF_EINVAL;
  return dev_rc(read_launch(src, (size_t)bytes, sink, (hipStream_t)stream));
}

}  // extern "C"
