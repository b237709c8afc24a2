// HIP executor of one continuous-batched iteration (chunked prefill + paged
// decode + greedy sampling) of a Llama-style decoder.
#include "executor.hpp"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <unordered_set>

#include "decode_plan.hpp"
#include "kernels/kernels.hpp"

namespace hxf {

namespace {

constexpr int kMaxSplits = 8;


// memcpy of a vector's elements; nothing for an empty one (whose data() may be null)
template <typename T>
void copy_vec(void* dst, const std::vector<T>& v) {
  if (!v.empty()) std::memcpy(dst, v.data(), v.size() * sizeof(T));
}

int64_t align256(int64_t x) { return (x + 255) & ~int64_t(255); }

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

#define HXF_HIP(call)                                                           \
  do {                                                                          \
    hipError_t e_ = (call);                                                     \
    if (e_ != hipSuccess) {                                                     \
      err = std::string("hip: ") + #call + ": " + hipGetErrorString(e_);        \
      return HXF_EDEVICE;                                                       \
    }                                                                           \
  } while (0)

}  // namespace

int validate_model(const hxf_model_cfg& m, std::string& err) {
  if (m.n_layers <= 0 || m.d_model <= 0 || m.n_q_heads <= 0 || m.n_kv_heads <= 0 || m.ffn_dim <= 0 ||
      m.vocab <= 0 || m.max_context <= 0) {
    err = "model: sizes must be positive";
    return HXF_EINVAL;
  }
  if (m.page_size != kPage) { err = "model: page_size must be 16"; return HXF_EINVAL; }
  if (m.head_dim != 64 && m.head_dim != 128) { err = "model: head_dim must be 64 or 128"; return HXF_EINVAL; }
  if (m.n_q_heads % m.n_kv_heads != 0 || m.n_q_heads / m.n_kv_heads > 16) {
    err = "model: n_q_heads must be a multiple of n_kv_heads, group <= 16";
    return HXF_EINVAL;
  }
  if (m.d_model % 64 != 0 || m.ffn_dim % 16 != 0 || m.vocab % 8 != 0) {
    err = "model: d_model % 64, ffn_dim % 16 and vocab % 8 must be 0";
    return HXF_EINVAL;
  }
  if (!(m.rms_eps > 0.f) || !(m.rope_base > 1.f)) { err = "model: bad eps or rope base"; return HXF_EINVAL; }
  return HXF_OK;
}

int64_t kv_pool_bytes(const hxf_model_cfg& m, int64_t n_blocks) {
  return (int64_t)m.n_layers * 2 * n_blocks * m.n_kv_heads * kPage * m.head_dim * 2;
}

WsPlan plan_workspace(const hxf_model_cfg& m, const hxf_sched_cfg& s) {
  WsPlan p;
  const int64_t d = m.d_model, dh = m.head_dim, hq = m.n_q_heads, hkv = m.n_kv_heads, f = m.ffn_dim;
  const int64_t G = hq / hkv;
  const int64_t qkv = (hq + 2 * hkv) * dh;
  p.t_max = (int64_t)s.chunk_tokens + s.max_seqs;
  p.r_max = s.max_seqs;
  p.e_max = s.max_seqs;
  p.bt_w = ceil_div(m.max_context, kPage);
  p.dec_items_max = decode_parts_bound(s.max_seqs, hkv, m.max_context);
  p.merges_max = (int64_t)s.max_seqs * hkv;
  const int qpi = prefill_queries_per_item((int)G);
  p.pf_merges_max = hkv * (ceil_div(s.chunk_tokens, qpi) + s.max_seqs);   // whole prefill items
  p.pf_parts_max = prefill_parts_bound(p.pf_merges_max);
  p.pf_items_max = p.pf_merges_max + kPrefillResident;                    // with the parts of split items
  // metadata (int32 words), sections packed in this order, each 64-word aligned
  auto words = [](int64_t n) { return (n + 63) & ~int64_t(63); };
  const int64_t meta_words = words(1) + words(p.t_max) * 3 + words(p.r_max) + words(p.e_max) * 2 +
                             words(p.e_max * p.bt_w) + words(p.dec_items_max * (int64_t)(sizeof(DecodeItem) / 4)) +
                             words(p.merges_max * 4) + words(p.pf_items_max * (int64_t)(sizeof(PrefillItem) / 4)) +
                             words(p.pf_merges_max * (int64_t)(sizeof(PrefillMerge) / 4));
  p.meta_bytes = meta_words * 4;
  // split-K partials: largest splits*M*N over the GEMM shapes at M <= 512 (no plan
  // splits K above 512 rows)
  int64_t part = 0;
  const int64_t shapes[5][3] = {{qkv, d, 0}, {d, hq * dh, 0}, {2 * f, d, 1}, {d, f, 0}, {m.vocab, d, 0}};
  for (int64_t M = 1; M <= std::min<int64_t>(512, p.t_max); ++M)
    for (auto& sh : shapes) {
      GemmPlan g = gemm_plan((int)M, (int)sh[0], (int)sh[1], kMaxSplits, sh[2] != 0);
      if (g.splits > 1) part = std::max(part, (int64_t)g.splits * M * sh[0] * 4);
    }
  int64_t o = 0;
  auto take = [&](int64_t bytes) { int64_t at = o; o = align256(o + bytes); return at; };
  p.off_meta = take(p.meta_bytes);
  p.off_rope = take((int64_t)m.max_context * (dh / 2) * 8);
  p.off_resid = take(p.t_max * d * 4);
  // the GEMM activations are stored in the packed tile layout: whole 16-row tiles
  const int64_t t16 = (p.t_max + 15) / 16 * 16;
  p.off_h = take(t16 * d * 2);
  p.off_qkv = take(p.t_max * qkv * 2);
  p.off_attn = take(t16 * hq * dh * 2);
  p.off_act = take(t16 * f * 2);
  p.part_bytes = part;
  p.off_part = take(std::max<int64_t>(part, 256));
  p.off_attn_o = take(p.dec_items_max * G * dh * 4);
  p.off_attn_ml = take(p.dec_items_max * G * 2 * 4);
  p.off_pf_o = take(p.pf_parts_max * kPrefillPairs * dh * 4);
  p.off_pf_ml = take(p.pf_parts_max * kPrefillPairs * 2 * 4);
  p.off_logits = take(p.r_max * m.vocab * 4);
  p.off_hr = take(p.r_max * d * 2);
  p.off_sampled = take(p.r_max * 4);
  p.total = o;
  return p;
}

void build_rope_table(std::vector<float>& out, int max_pos, int dh, float base) {
  const int half = dh / 2;
  out.resize((size_t)max_pos * half * 2);
  for (int i = 0; i < half; ++i) {
    const double theta = std::pow((double)base, -2.0 * i / dh);
    for (int p = 0; p < max_pos; ++p) {
      const double a = (double)p * theta;
      out[((size_t)p * half + i) * 2] = (float)std::cos(a);
      out[((size_t)p * half + i) * 2 + 1] = (float)std::sin(a);
    }
  }
}

namespace {

class HipExecutor : public Executor {
 public:
  HipExecutor(const hxf_model_cfg& m, const hxf_sched_cfg& s, const hxf_device_buffers& b, void* stream)
      : m_(m), s_(s), b_(b), st_((hipStream_t)stream) {
    layers_.assign(b.layers, b.layers + m.n_layers);
    plan_ = plan_workspace(m, s);
    ws_ = reinterpret_cast<uint8_t*>(b.workspace);
    const char* ng = std::getenv("HXF_NO_GRAPHS");
    use_graphs_ = !(ng && ng[0] && ng[0] != '0');
    const char* ck = std::getenv("HXF_CHECK");
    check_ = ck && ck[0] && ck[0] != '0';
  }

  ~HipExecutor() override {
    drop_graphs();
    if (graph_st_) (void)hipStreamDestroy(graph_st_);
    if (host_meta_) (void)hipHostFree(host_meta_);
    if (host_sampled_) (void)hipHostFree(host_sampled_);
    if (ev_) {
      for (auto& e : ev_pool_) (void)hipEventDestroy(e);
    }
  }

  int init(std::string& err) {
    HXF_HIP(hipHostMalloc(&host_meta_, plan_.meta_bytes, hipHostMallocDefault));
    HXF_HIP(hipHostMalloc(reinterpret_cast<void**>(&host_sampled_), plan_.r_max * 4, hipHostMallocDefault));
    std::vector<float> tab;
    build_rope_table(tab, m_.max_context, m_.head_dim, m_.rope_base);
    HXF_HIP(hipMemcpyAsync(ws_ + plan_.off_rope, tab.data(), tab.size() * 4, hipMemcpyHostToDevice, st_));
    HXF_HIP(hipStreamSynchronize(st_));
    ev_ = true;
    return HXF_OK;
  }

  int run(const std::vector<BatchEntry>& batch, std::vector<int32_t>& sampled, std::string& err) override;
  int last_logits(uint64_t id, float* dst, int32_t cap, std::string& err) override;

  Profile prof;

 private:
  template <typename T>
  T* dev(int64_t off) { return reinterpret_cast<T*>(ws_ + off); }
  // With `pending` set, a split-K plan leaves its partials in the workspace and
  // *pending = its split count (0 when the GEMM finished its own epilogue).
  // `kind` (HXF_PROF_*) names the projection for profiling.
  // a_packed: A in the packed tile layout; c_kt > 0: the SwiGLU output packed.
  int gemm(const uint16_t* A, int lda, const uint16_t* B, const uint16_t* B2, void* C, int ldc, int M, int N, int K,
           int epi, int kind, std::string& err, int* pending = nullptr, bool a_packed = false, int c_kt = 0);
  // A pair of events for a profiled launch of `kind` (0-4 GEMMs, 5 prefill attention)
  // doing `flops`; null events when profiling is off.
  int prof_events(int kind, double flops, hipEvent_t* e0, hipEvent_t* e1, std::string& err);
  struct ProfEv {
    int kind;
    hipEvent_t e0, e1;
    double flops;
  };
  std::vector<ProfEv> prof_ev_;

  hxf_model_cfg m_;
  hxf_sched_cfg s_;
  hxf_device_buffers b_;
  hipStream_t st_;
  std::vector<hxf_layer_weights> layers_;
  WsPlan plan_;
  uint8_t* ws_ = nullptr;
  void* host_meta_ = nullptr;
  int32_t* host_sampled_ = nullptr;
  std::vector<uint64_t> last_rows_;   // request id per logits row of the last iteration
  DecodePlan dplan_;                  // decode-attention work list of the current iteration
  PrefillPlan pplan_;                 // prefill-attention work list of the current iteration
  bool ev_ = false;
  std::vector<hipEvent_t> ev_pool_, ev_merge_;
  // Decode-only iterations replay a captured HIP graph of the whole forward (metadata
  // upload, every kernel, sampled ids back), keyed by the batch's launch shape; the
  // graph reads the per-iteration metadata from the pinned staging buffer.  A shape is
  // captured the second time it occurs (a capture costs more than an eager launch, and
  // under continuous batching many shapes occur once); at most kMaxGraphs are kept,
  // the least recently used one is replaced.
  static constexpr size_t kMaxGraphs = 16, kMaxSeen = 4096;
  struct GraphRec {
    int64_t key = 0;
    hipGraphExec_t exec = nullptr;
    int64_t last_use = 0;
  };
  std::vector<GraphRec> graphs_;
  std::unordered_set<int64_t> seen_;   // shapes met once, not captured yet
  int64_t graph_clock_ = 0;
  bool use_graphs_ = true;
  bool check_ = false;   // HXF_CHECK: validate every index the kernels will follow before launching
  // The legacy null stream cannot be captured: graphs then run on a stream of our own
  // (blocking, default priority), which the null stream orders against.
  hipStream_t graph_st_ = nullptr;
  void drop_graphs() {
    for (auto& g : graphs_)
      if (g.exec) (void)hipGraphExecDestroy(g.exec);
    graphs_.clear();
    seen_.clear();
  }
};

int HipExecutor::prof_events(int kind, double flops, hipEvent_t* e0, hipEvent_t* e1, std::string& err) {
  *e0 = *e1 = nullptr;
  if (!prof.on) return HXF_OK;
  HXF_HIP(hipEventCreate(e0));
  HXF_HIP(hipEventCreate(e1));
  prof_ev_.push_back(ProfEv{kind, *e0, *e1, flops});
  return HXF_OK;
}

int HipExecutor::gemm(const uint16_t* A, int lda, const uint16_t* B, const uint16_t* B2, void* C, int ldc, int M,
                      int N, int K, int epi, int kind, std::string& err, int* pending, bool a_packed, int c_kt) {
  GemmArgs a{};
  a.a_packed = a_packed ? 1 : 0;
  a.c_kt = c_kt;
  a.A = A;
  a.B = B;
  a.B2 = B2;
  a.C = C;
  a.partial = dev<float>(plan_.off_part);
  a.M = M;
  a.N = N;
  a.K = K;
  a.lda = lda;
  a.ldc = ldc;
  a.kt = (K + 31) / 32;
  GemmPlan p = gemm_plan(M, N, K, kMaxSplits, epi == EPI_SWIGLU);
  if (p.splits > 1 && (int64_t)p.splits * M * N * 4 > plan_.part_bytes) {
    err = "gemm: split-K partial buffer too small";
    return HXF_EINVAL;
  }
  const bool defer = pending && p.splits > 1;
  hipEvent_t e0, e1;
  if (int rc = prof_events(kind, 2.0 * M * N * K, &e0, &e1, err)) return rc;
  HXF_HIP(gemm_launch(a, epi, p, st_, !defer, e0, e1));
  if (pending) *pending = defer ? p.splits : 0;
  return HXF_OK;
}

int HipExecutor::run(const std::vector<BatchEntry>& batch, std::vector<int32_t>& sampled, std::string& err) {
  const int E = (int)batch.size();
  const int d = m_.d_model, dh = m_.head_dim, hq = m_.n_q_heads, hkv = m_.n_kv_heads, f = m_.ffn_dim;
  const int G = hq / hkv;
  const int qkv_w = (hq + 2 * hkv) * dh;
  int T = 0, R = 0, n_dec = 0, bt_w = 1;
  for (const auto& e : batch) {
    T += e.n;
    R += e.logits ? 1 : 0;
    n_dec += e.decode ? 1 : 0;
    bt_w = std::max<int>(bt_w, (int)ceil_div((int64_t)e.pos0 + e.n, kPage));
  }
  if (T > plan_.t_max || R > plan_.r_max || E > plan_.e_max) {
    err = "run: batch exceeds the workspace plan";
    return HXF_EINVAL;
  }
  // ---------------------------------------------------------- metadata
  // A decode-only batch uses a layout that depends only on its launch shape (E rows,
  // block tables padded to a multiple of 64 pages, a fixed work-item capacity), so that
  // its forward can be captured once and replayed; the decode-attention grid is then
  // that capacity and the kernel reads the real item count from the metadata.
  // (Profiling stamps the attention kernels' own start and end, which a captured graph
  // cannot, so profiled iterations launch eagerly.)
  const bool pure_decode = E > 0 && n_dec == E;
  const bool graph = pure_decode && use_graphs_ && !prof.on;
  if (graph) bt_w = (int)std::min<int64_t>(plan_.bt_w, ((bt_w + 63) / 64) * 64);
  const int64_t item_cap =
      graph ? std::min<int64_t>(plan_.dec_items_max, std::max<int64_t>(kDecodeResident, 2LL * E * hkv)) : 0;
  int32_t* hm = reinterpret_cast<int32_t*>(host_meta_);
  int64_t w = 0;
  auto sec = [&](int64_t n) { int64_t at = w; w += (n + 63) & ~int64_t(63); return at; };
  const int64_t o_nitems = sec(2);
  const int64_t o_ids = sec(T), o_pos = sec(T), o_slot = sec(T), o_lrow = sec(R), o_row0 = sec(E), o_pos0 = sec(E),
                o_bt = sec((int64_t)E * bt_w);
  int row = 0, r = 0;
  std::vector<DecodeSeq> dseqs;
  dseqs.reserve(n_dec);
  std::vector<PrefillEntry> pentries;
  const int qpi = prefill_queries_per_item(G);
  last_rows_.clear();
  for (int e = 0; e < E; ++e) {
    const BatchEntry& be = batch[e];
    const std::vector<int32_t>& bt = be.r->bt;
    for (int k = 0; k < be.n; ++k) {
      const int p = be.pos0 + k;
      hm[o_ids + row + k] = be.toks[k];
      hm[o_pos + row + k] = p;
      hm[o_slot + row + k] = bt[p / kPage] * kPage + p % kPage;
    }
    if (be.logits) {
      hm[o_lrow + r++] = row + be.n - 1;
      last_rows_.push_back(be.r->id);
    }
    hm[o_row0 + e] = row;
    hm[o_pos0 + e] = be.pos0;
    const int np = (int)ceil_div((int64_t)be.pos0 + be.n, kPage);
    for (int j = 0; j < bt_w; ++j) hm[o_bt + (int64_t)e * bt_w + j] = j < np ? bt[j] : 0;
    if (be.decode) {
      dseqs.push_back(DecodeSeq{e, be.pos0 + 1, bt.data()});
    } else {
      pentries.push_back(PrefillEntry{e, be.pos0, be.n});
    }
    row += be.n;
  }
  plan_prefill(pentries, hkv, qpi, pplan_);
  const std::vector<PrefillItem>& pitems = pplan_.items;
  const std::vector<PrefillMerge>& pmerges = pplan_.merges;
  plan_decode(dseqs, hkv, G, dplan_);
  const std::vector<DecodeItem>& ditems = dplan_.items;
  const std::vector<MergeItem>& merges = dplan_.merges;
  if (dplan_.n_wide < 0 || dplan_.n_wide > (int64_t)ditems.size()) {
    err = "run: decode work list counts are inconsistent";
    return HXF_EINVAL;
  }
  if ((int64_t)ditems.size() > plan_.dec_items_max || dplan_.n_parts > plan_.dec_items_max ||
      (int64_t)pitems.size() > plan_.pf_items_max || (int64_t)pmerges.size() > plan_.pf_merges_max ||
      pplan_.n_parts > plan_.pf_parts_max || (graph && (int64_t)ditems.size() > item_cap)) {
    err = "run: attention work list exceeds the workspace plan";
    return HXF_EINVAL;
  }
  constexpr int64_t kItemWords = sizeof(DecodeItem) / 4;
  const int64_t o_ditems = sec((graph ? item_cap : (int64_t)ditems.size()) * kItemWords),
                o_merges = sec((int64_t)merges.size() * 4),
                o_pitems = sec((int64_t)pitems.size() * (int64_t)(sizeof(PrefillItem) / 4)),
                o_pmerges = sec((int64_t)pmerges.size() * (int64_t)(sizeof(PrefillMerge) / 4));
  if (w * 4 > plan_.meta_bytes) {
    err = "run: metadata exceeds the workspace plan";
    return HXF_EINVAL;
  }
  const int64_t n_wide = dplan_.n_wide, n_narrow = (int64_t)ditems.size() - n_wide;
  hm[o_nitems] = (int32_t)n_narrow;
  hm[o_nitems + 1] = (int32_t)n_wide;
  copy_vec(hm + o_ditems, ditems);
  copy_vec(hm + o_merges, merges);
  copy_vec(hm + o_pitems, pitems);
  copy_vec(hm + o_pmerges, pmerges);
  if (check_) {
    // every index a kernel follows, checked on the host against the buffers it addresses
    auto fail = [&](const char* what, int64_t i) {
      err = std::string("check: ") + what + " (index " + std::to_string(i) + ")";
      return HXF_EINVAL;
    };
    const int64_t slots = s_.n_blocks * kPage;
    for (int64_t i = 0; i < T; ++i) {
      if (hm[o_ids + i] < 0 || hm[o_ids + i] >= m_.vocab) return fail("token id outside the vocabulary", i);
      if (hm[o_pos + i] < 0 || hm[o_pos + i] >= m_.max_context) return fail("position outside max_context", i);
      if (hm[o_slot + i] < 0 || hm[o_slot + i] >= slots) return fail("KV slot outside the pool", i);
    }
    for (int i = 0; i < R; ++i)
      if (hm[o_lrow + i] < 0 || hm[o_lrow + i] >= T) return fail("logits row outside the batch", i);
    std::vector<int32_t> ctx(E);
    for (int e = 0; e < E; ++e) {
      ctx[e] = batch[e].pos0 + batch[e].n;
      const int64_t np = ceil_div((int64_t)ctx[e], kPage);
      if (np > bt_w) return fail("block table wider than its stride", e);
      for (int64_t j = 0; j < np; ++j) {
        const int32_t b = hm[o_bt + (int64_t)e * bt_w + j];
        if (b < 0 || b >= s_.n_blocks) return fail("block-table entry outside the pool", e);
      }
    }
    for (size_t i = 0; i < ditems.size(); ++i) {
      const DecodeItem& d = ditems[i];
      const int rows_max = (int64_t)i < n_narrow ? decode_rows_narrow(G) : decode_rows_wide(G);
      if (d.kvh < 0 || d.kvh >= hkv || d.t0 < 0 || d.t0 >= d.t1 || d.n_rows < 1 || d.n_rows > rows_max)
        return fail("decode item", (int64_t)i);
      for (int k = 0; k < d.n_rows; ++k)
        if (d.entry[k] < 0 || d.entry[k] >= E || !batch[d.entry[k]].decode || d.t1 > ctx[d.entry[k]] ||
            d.part[k] < 0 || d.part[k] >= dplan_.n_parts)
          return fail("decode item row", (int64_t)i);
    }
    for (size_t i = 0; i < merges.size(); ++i) {
      const MergeItem& mi = merges[i];
      if (mi.entry < 0 || mi.entry >= E || mi.kvh < 0 || mi.kvh >= hkv || mi.n_part < 1 || mi.part0 < 0 ||
          mi.part0 + mi.n_part > dplan_.n_parts)
        return fail("merge item", (int64_t)i);
    }
    for (size_t i = 0; i < pitems.size(); ++i) {
      const PrefillItem& pi = pitems[i];
      if (pi.entry < 0 || pi.entry >= E || batch[pi.entry].decode || pi.kvh < 0 || pi.kvh >= hkv || pi.q0 < 0 ||
          pi.nq < 1 || pi.nq * G > kPrefillPairs || pi.q0 + pi.nq > batch[pi.entry].n || pi.t0 < 0 ||
          pi.t0 >= pi.t1 || (int64_t)pi.t1 * 32 > ((int64_t)ctx[pi.entry] + 31) / 32 * 32 ||
          pi.part >= pplan_.n_parts)
        return fail("prefill item", (int64_t)i);
    }
    for (size_t i = 0; i < pmerges.size(); ++i) {
      const PrefillMerge& pm = pmerges[i];
      if (pm.entry < 0 || pm.entry >= E || batch[pm.entry].decode || pm.kvh < 0 || pm.kvh >= hkv || pm.nq < 1 ||
          pm.nq * G > kPrefillPairs || pm.q0 < 0 || pm.q0 + pm.nq > batch[pm.entry].n || pm.n_part < 1 ||
          pm.part0 < 0 || pm.part0 + pm.n_part > pplan_.n_parts)
        return fail("prefill merge", (int64_t)i);
    }
  }
  int32_t* dm = dev<int32_t>(plan_.off_meta);

  // ---------------------------------------------------------- forward
  float* resid = dev<float>(plan_.off_resid);
  uint16_t* h = dev<uint16_t>(plan_.off_h);
  uint16_t* qkv = dev<uint16_t>(plan_.off_qkv);
  uint16_t* attn = dev<uint16_t>(plan_.off_attn);
  uint16_t* act = dev<uint16_t>(plan_.off_act);
  const float2* rope = dev<float2>(plan_.off_rope);
  const float scale_log2 = 1.4426950408889634f / std::sqrt((float)dh);
  // The GEMM activations (the normed hidden state, the attention output, the SwiGLU output)
  // are kept in the packed tile layout of the weights, in which a 16 x 32 block the GEMMs
  // stage is one contiguous kilobyte rather than 16 row pieces, when the widths allow it.
  const bool pack = d % 32 == 0 && f % 32 == 0 && (hq * dh) % 32 == 0;
  const int kt_h = pack ? d / 32 : 0, kt_attn = pack ? hq * dh / 32 : 0, kt_act = pack ? f / 32 : 0;
  const int64_t layer_pool = (int64_t)s_.n_blocks * hkv * kPage * dh;   // bf16 elements per K (or V) pool
  uint16_t* pool = reinterpret_cast<uint16_t*>(b_.kv_pool);

  DecodeAttnArgs da{};
  da.q = qkv;
  da.q_row = dm + o_row0;
  da.q_stride = qkv_w;
  da.n_blocks = s_.n_blocks;
  da.bt = dm + o_bt;
  da.bt_stride = bt_w;
  da.items = reinterpret_cast<const DecodeItem*>(dm + o_ditems);
  da.n_items = graph ? (int)item_cap : (int)n_narrow;
  da.n_wide = graph ? (n_wide ? (int)item_cap : 0) : (int)n_wide;
  da.n_items_dev = graph ? dm + o_nitems : nullptr;
  da.merges = reinterpret_cast<const MergeItem*>(dm + o_merges);
  da.n_merges = (int)merges.size();
  da.part_o = dev<float>(plan_.off_attn_o);
  da.part_ml = dev<float>(plan_.off_attn_ml);
  da.out = attn;
  da.out_stride = hq * dh;
  da.out_kt = kt_attn;
  da.Hq = hq;
  da.Hkv = hkv;
  da.dh = dh;
  da.scale_log2 = scale_log2;
  PrefillAttnArgs pa{};
  pa.q = qkv;
  pa.q_stride = qkv_w;
  pa.n_blocks = s_.n_blocks;
  pa.row0 = dm + o_row0;
  pa.pos0 = dm + o_pos0;
  pa.bt = dm + o_bt;
  pa.bt_stride = bt_w;
  pa.items = reinterpret_cast<const PrefillItem*>(dm + o_pitems);
  pa.n_items = (int)pitems.size();
  pa.merges = reinterpret_cast<const PrefillMerge*>(dm + o_pmerges);
  pa.n_merges = (int)pmerges.size();
  pa.part_o = dev<float>(plan_.off_pf_o);
  pa.part_ml = dev<float>(plan_.off_pf_ml);
  pa.out = attn;
  pa.out_stride = hq * dh;
  pa.out_kt = kt_attn;
  pa.Hq = hq;
  pa.Hkv = hkv;
  pa.dh = dh;
  pa.scale_log2 = scale_log2;

  const int64_t kv_tokens = dplan_.kv_tokens;
  // prefill attention work: 4*dh flops per (query, visible key, q-head)
  double pf_attn_flops = 0;
  for (const auto& be : batch)
    if (!be.decode) pf_attn_flops += ((double)be.n * be.pos0 + 0.5 * be.n * (be.n + 1.0)) * hq * 4.0 * dh;
  uint16_t* hr = dev<uint16_t>(plan_.off_hr);
  float* logits = dev<float>(plan_.off_logits);
  int32_t* samp = dev<int32_t>(plan_.off_sampled);

  // The launch sequence (eager, or recorded by a stream capture).
  auto forward = [&]() -> int {
    HXF_HIP(hipMemcpyAsync(dm, hm, w * 4, hipMemcpyHostToDevice, st_));
    HXF_HIP(embed_rmsnorm_launch(dm + o_ids, (const uint16_t*)b_.embed, (const uint16_t*)layers_[0].attn_norm,
                                 resid, h, T, d, m_.rms_eps, st_, kt_h));
    // Split-K GEMMs of decode-sized batches hand their partials to the next kernel
    // (RoPE/KV write, residual add + RMSNorm), which sums them in split order.
    float* part = dev<float>(plan_.off_part);
    int pend_down = 0;
    for (int l = 0; l < m_.n_layers; ++l) {
      const hxf_layer_weights& L = layers_[l];
      uint16_t* kp = pool + (int64_t)l * 2 * layer_pool;
      uint16_t* vp = kp + layer_pool;
      if (l > 0)
        HXF_HIP(resid_rmsnorm_launch(resid, part, pend_down, T, nullptr, (const uint16_t*)L.attn_norm, h, T, d,
                                     m_.rms_eps, st_, kt_h));
      int pend_qkv = 0;
      if (int rc = gemm(h, d, (const uint16_t*)L.wqkv, nullptr, qkv, qkv_w, T, qkv_w, d, EPI_BF16, HXF_PROF_QKV, err,
                        &pend_qkv, pack))
        return rc;
      if (pend_qkv)
        HXF_HIP(rope_kv_partials_launch(qkv, part, pend_qkv, dm + o_pos, dm + o_slot, rope, kp, vp, s_.n_blocks, T, hq,
                                        hkv, dh, st_));
      else
        HXF_HIP(rope_kv_launch(qkv, dm + o_pos, dm + o_slot, rope, kp, vp, s_.n_blocks, T, hq, hkv, dh, st_));
      da.k_pool = pa.k_pool = kp;
      da.v_pool = pa.v_pool = vp;
      if (da.n_items || da.n_wide) {
        hipEvent_t e0 = nullptr, e1 = nullptr, e2 = nullptr, e3 = nullptr;
        if (prof.on) {
          HXF_HIP(hipEventCreate(&e0));
          HXF_HIP(hipEventCreate(&e1));
          HXF_HIP(hipEventCreate(&e2));
          HXF_HIP(hipEventCreate(&e3));
        }
        HXF_HIP(decode_attn_launch(da, st_, e0, e1));
        HXF_HIP(decode_merge_launch(da, st_, e2, e3));
        if (prof.on) {
          ev_pool_.push_back(e0);
          ev_pool_.push_back(e1);
          ev_merge_.push_back(e2);
          ev_merge_.push_back(e3);
        }
      }
      if (pa.n_items) {
        hipEvent_t e0, e1;
        if (int rc = prof_events(5, pf_attn_flops, &e0, &e1, err)) return rc;
        HXF_HIP(prefill_attn_launch(pa, st_, e0, e1));
      }
      int pend_o = 0;
      if (int rc =
              gemm(attn, hq * dh, (const uint16_t*)L.wo, nullptr, resid, d, T, d, hq * dh, EPI_RESID, HXF_PROF_O, err,
                   &pend_o, pack))
        return rc;
      HXF_HIP(resid_rmsnorm_launch(resid, part, pend_o, T, nullptr, (const uint16_t*)L.ffn_norm, h, T, d, m_.rms_eps,
                                   st_, kt_h));
      if (int rc =
              gemm(h, d, (const uint16_t*)L.w_gate, (const uint16_t*)L.w_up, act, f, T, 2 * f, d, EPI_SWIGLU,
                   HXF_PROF_GATE_UP, err, nullptr, pack, kt_act))
        return rc;
      if (int rc = gemm(act, f, (const uint16_t*)L.w_down, nullptr, resid, d, T, d, f, EPI_RESID, HXF_PROF_DOWN, err,
                        &pend_down, pack))
        return rc;
    }
    if (R > 0) {
      // (rows without logits never need the last down projection's partials)
      HXF_HIP(resid_rmsnorm_launch(resid, part, pend_down, T, dm + o_lrow, (const uint16_t*)b_.final_norm, hr, R, d,
                                   m_.rms_eps, st_));
      if (int rc = gemm(hr, d, (const uint16_t*)b_.lm_head, nullptr, logits, m_.vocab, R, m_.vocab, d, EPI_F32,
                           HXF_PROF_LM_HEAD, err))
        return rc;
      HXF_HIP(argmax_launch(logits, samp, R, m_.vocab, st_));
      HXF_HIP(hipMemcpyAsync(host_sampled_, samp, (size_t)R * 4, hipMemcpyDeviceToHost, st_));
    }
    return HXF_OK;
  };

  if (!graph) {
    if (int rc = forward()) return rc;
    HXF_HIP(hipStreamSynchronize(st_));
  } else {
    // every launch of forward() goes to st_: point it at the capture stream meanwhile
    struct StreamSwap {
      hipStream_t& ref;
      hipStream_t saved;
      ~StreamSwap() { ref = saved; }
    } swap{st_, st_};
    if (!st_) {
      if (!graph_st_) HXF_HIP(hipStreamCreate(&graph_st_));
      st_ = graph_st_;
    }
    const int64_t key = ((int64_t)E << 32) | ((int64_t)bt_w << 1) | (dplan_.n_wide > 0 ? 1 : 0);
    GraphRec* g = nullptr;
    for (auto& x : graphs_)
      if (x.key == key) g = &x;
    const bool capture = !g && !seen_.insert(key).second;   // second occurrence of the shape
    if (capture) {
      seen_.erase(key);
      if (seen_.size() > kMaxSeen) seen_.clear();
      if (graphs_.size() >= kMaxGraphs) {
        auto lru = std::min_element(graphs_.begin(), graphs_.end(),
                                    [](const GraphRec& a, const GraphRec& b) { return a.last_use < b.last_use; });
        if (lru->exec) (void)hipGraphExecDestroy(lru->exec);
        graphs_.erase(lru);
      }
      GraphRec rec;
      rec.key = key;
      HXF_HIP(hipStreamBeginCapture(st_, hipStreamCaptureModeThreadLocal));
      const int rc = forward();
      hipGraph_t cg = nullptr;
      const hipError_t ec = hipStreamEndCapture(st_, &cg);
      hipError_t ei = hipSuccess;
      if (rc == HXF_OK && ec == hipSuccess) ei = hipGraphInstantiate(&rec.exec, cg, nullptr, nullptr, 0);
      if (cg) (void)hipGraphDestroy(cg);
      if (rc != HXF_OK) return rc;
      if (ec != hipSuccess || ei != hipSuccess) {
        // the runtime could not capture or instantiate: stop using graphs, launch eagerly
        (void)hipGetLastError();
        if (rec.exec) (void)hipGraphExecDestroy(rec.exec);
        use_graphs_ = false;
      } else {
        graphs_.push_back(std::move(rec));
        g = &graphs_.back();
      }
    }
    if (g) {
      g->last_use = ++graph_clock_;
      HXF_HIP(hipGraphLaunch(g->exec, st_));
    } else if (int rc = forward()) {
      return rc;
    }
    HXF_HIP(hipStreamSynchronize(st_));
  }
  if (prof.on && (da.n_items || da.n_wide)) {
    prof.decode_attn_launches += m_.n_layers;
    prof.decode_attn_bytes += (int64_t)m_.n_layers * kv_tokens * 2 * dh * 2;
  }
  if (prof.on) {
    for (size_t i = 0; i + 1 < ev_pool_.size(); i += 2) {
      float ms = 0.f;
      HXF_HIP(hipEventElapsedTime(&ms, ev_pool_[i], ev_pool_[i + 1]));
      prof.decode_attn_ms += ms;
      (void)hipEventDestroy(ev_pool_[i]);
      (void)hipEventDestroy(ev_pool_[i + 1]);
    }
    ev_pool_.clear();
    for (size_t i = 0; i + 1 < ev_merge_.size(); i += 2) {
      float ms = 0.f;
      HXF_HIP(hipEventElapsedTime(&ms, ev_merge_[i], ev_merge_[i + 1]));
      prof.decode_merge_ms += ms;
      (void)hipEventDestroy(ev_merge_[i]);
      (void)hipEventDestroy(ev_merge_[i + 1]);
    }
    ev_merge_.clear();
    for (const ProfEv& pe : prof_ev_) {
      float ms = 0.f;
      HXF_HIP(hipEventElapsedTime(&ms, pe.e0, pe.e1));
      if (pe.kind < 5) {
        prof.gemm_launches[pe.kind] += 1;
        prof.gemm_flops[pe.kind] += pe.flops;
        prof.gemm_ms[pe.kind] += ms;
      } else {
        prof.prefill_attn_launches += 1;
        prof.prefill_attn_flops += pe.flops;
        prof.prefill_attn_ms += ms;
      }
      (void)hipEventDestroy(pe.e0);
      (void)hipEventDestroy(pe.e1);
    }
    prof_ev_.clear();
  }
  sampled.assign(host_sampled_, host_sampled_ + R);
  return HXF_OK;
}

int HipExecutor::last_logits(uint64_t id, float* dst, int32_t cap, std::string& err) {
  for (size_t i = 0; i < last_rows_.size(); ++i) {
    if (last_rows_[i] != id) continue;
    if (cap < m_.vocab) {
      err = "last_logits: buffer smaller than vocab";
      return HXF_ENOMEM;
    }
    HXF_HIP(hipMemcpyAsync(dst, dev<float>(plan_.off_logits) + i * (size_t)m_.vocab, (size_t)m_.vocab * 4,
                           hipMemcpyDeviceToHost, st_));
    HXF_HIP(hipStreamSynchronize(st_));
    return HXF_OK;
  }
  err = "last_logits: request had no logits row in the last iteration";
  return HXF_ENOTFOUND;
}

}  // namespace

std::unique_ptr<Executor> make_hip_executor(const hxf_model_cfg& m, const hxf_sched_cfg& s,
                                            const hxf_device_buffers& b, void* stream, std::string& err, int* rc) {
  auto ex = std::make_unique<HipExecutor>(m, s, b, stream);
  *rc = ex->init(err);
  if (*rc) return nullptr;
  return ex;
}

Profile* executor_profile(Executor* e) {
  auto* h = dynamic_cast<HipExecutor*>(e);
  return h ? &h->prof : nullptr;
}

}  // namespace hxf
