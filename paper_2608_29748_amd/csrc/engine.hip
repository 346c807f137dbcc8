// Host runtime of the ReTrace round: workspace carving, weight packing, prefill,
// the round's kernel sequence (captured once into a HIP graph), and the C ABI.
#include <hip/hip_runtime.h>
#include <math.h>
#include <string.h>

#include <mutex>
#include <new>
#include <vector>

#include "attn.h"
#include "gemm.h"
#include "host.h"
#include "misc.h"
#include "sample.h"

namespace rt {
const char* last_error();

// Static scratch of the allocation-free round (rt_spec_round_static): the partial
// results of its kernels (GEMM split partials and split-K arrival counters, residual
// k-slab partials, attention key-split partials and plan).  Each GPU the library runs
// on holds its own copy until the process ends; host code reaches it only through the
// device address that hipGetSymbolAddress returns for the current device (the array's
// name is a host-side stand-in).  Every allocation-free round on a GPU shares it.
static __device__ __align__(256) char scratch[kStaticScratchBytes];
constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's static scratch, looked up once per device.
static int scratch_setup(int dev, void** out) {
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (dev < 0 || dev >= kMaxDevices) return fail(RT_ERR_HIP, "device %d outside the static scratch table", dev);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) return fail(RT_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return RT_OK;
}
LaunchEvents& launch_events() {
  static thread_local LaunchEvents ev;
  return ev;
}

#define HIPCHK(x)                                                                          \
  do {                                                                                     \
    hipError_t e_ = (x);                                                                   \
    if (e_ != hipSuccess) return fail(RT_ERR_HIP, "%s: %s", #x, hipGetErrorString(e_));    \
  } while (0)
#define CHK(x)                 \
  do {                         \
    int s_ = (x);              \
    if (s_ != RT_OK) return s_; \
  } while (0)

struct EngineBase {
  rt_config cfg{};
  Plan p{};
  char* ws = nullptr;
  int device = 0;                // the GPU the model was built on
  void* scratch_dev = nullptr;   // that GPU's static scratch (device address), or null
  int scratch_status = RT_OK;    // why scratch_dev is null
  // Partial-result buffers: in the workspace (part_base null), or from offset 0 of the
  // static scratch during rt_spec_round_static.
  char* part_base = nullptr;
  size_t part_off(size_t ws_off, size_t static_off) const { return part_base ? static_off : ws_off; }
  template <class X> X* pat(size_t ws_off, size_t static_off) const {
    return reinterpret_cast<X*>((part_base ? part_base : ws) + part_off(ws_off, static_off));
  }
  hipStream_t stream = nullptr;
  bool own_stream = false;
  int n_seqs = 0;
  bool prefilled = false;
  int flags = 0;
  hipGraph_t graph = nullptr;
  hipGraphExec_t gexec = nullptr;
  hipGraph_t ar_graph = nullptr;       // one target-only step
  hipGraphExec_t ar_gexec = nullptr;
  bool ar_mode = false;                // target-only steps ran since the last prefill
  int32_t* h_out = nullptr;      // pinned: tokens [R], n [bmax], a [bmax], first [bmax]
  // Layer trace (test hook, debug flag 8): the last eager round's intermediates of every
  // drafter and target layer, copied into a device buffer of its own.  One record per
  // layer (drafter layers 0..LD-1, then target layers), then one per pass for the
  // residual entering the final norm and the LM-head operand.  Items of a record: the
  // residual input (f32 [R][d]), q after its norm and RoPE ([R][qN]), the attention
  // output (packed operand), the residual after the attention block (f32), the
  // post-attention norm output (packed) and the SwiGLU product (packed).
  enum TraceItem { TI_X = 0, TI_Q, TI_ATTN, TI_XMID, TI_H2, TI_MLP, TI_COUNT };
  char* trace = nullptr;
  size_t trace_rec_bytes = 0;
  size_t trace_item_off[TI_COUNT] = {};
  size_t trace_item_bytes(int it) const {
    const size_t R = (size_t)p.R, R16 = rup((size_t)p.R, 16), E = (size_t)p.esz;
    switch (it) {
      case TI_X: case TI_XMID: return R * p.d * 4;
      case TI_Q: return R * p.qN * E;
      case TI_ATTN: return R16 * p.Kp_q * E;
      case TI_H2: return R16 * p.Kp_d * E;
      default: return R16 * p.Kp_F * E;
    }
  }
  bool tracing() const { return trace && (flags & 8) && !instrumented(); }
  int trace_item(int rec, int it, const void* src) {
    if (rec < 0 || !tracing()) return RT_OK;
    HIPCHK(hipMemcpyAsync(trace + (size_t)rec * trace_rec_bytes + trace_item_off[it], src, trace_item_bytes(it),
                          hipMemcpyDeviceToDevice, stream));
    return RT_OK;
  }
  int alloc_trace() {
    if (trace) return RT_OK;
    size_t off = 0;
    for (int it = 0; it < TI_COUNT; ++it) {
      trace_item_off[it] = off;
      off += rup(trace_item_bytes(it), 256);
    }
    trace_rec_bytes = off;
    HIPCHK(hipMalloc((void**)&trace, (size_t)(p.LD + p.L + 2) * trace_rec_bytes));
    return RT_OK;
  }
  // profiling: an event pair around every launch, aggregated per kernel kind
  bool profiling = false;
  std::vector<hipEvent_t> ev_pool;
  struct ProfRec { int kind; hipEvent_t b, e; double bytes, flops; };
  std::vector<ProfRec> prof;
  hipEvent_t stage_ev[RT_PROF_STAGES + 1] = {};
  std::vector<int32_t> prof_ctx;   // host copy of each sequence's context length
  size_t ev_next = 0;
  // kernel replay: only launches of this class are issued (and counted)
  int only_kind = -1;
  int only_launches = 0;
  double only_bytes = 0, only_flops = 0;
  bool instrumented() const { return profiling || only_kind >= 0; }
  // The next launch records the pair at its own start and end (see RT_LAUNCH).
  void prof_begin(int kind, double bytes, double flops) {
    if (only_kind >= 0) {
      const bool take = kind == only_kind;
      launch_events().skip = !take;
      if (take) { only_launches += 1; only_bytes += bytes; only_flops += flops; }
      return;
    }
    if (!profiling) return;
    ProfRec r{kind, ev_pool[ev_next], ev_pool[ev_next + 1], bytes, flops};
    ev_next += 2;
    prof.push_back(r);
    launch_events() = LaunchEvents{r.b, r.e, false};
  }
  void prof_end() {
    if (only_kind >= 0) { launch_events().skip = true; return; }
    if (!profiling) return;
    LaunchEvents& le = launch_events();
    if (!le.used) {   // nothing was launched: a zero-length record
      (void)hipEventRecord(prof.back().b, stream);
      (void)hipEventRecord(prof.back().e, stream);
    }
    le = LaunchEvents{};
  }
  void stage(int i) {
    if (profiling) (void)hipEventRecord(stage_ev[i], stream);
  }
  virtual ~EngineBase() {
    for (hipEvent_t e : ev_pool) (void)hipEventDestroy(e);
    for (hipEvent_t e : stage_ev) if (e) (void)hipEventDestroy(e);
    drop_graph();
    if (h_out) (void)hipHostFree(h_out);
    if (trace) (void)hipFree(trace);
    if (own_stream && stream) (void)hipStreamDestroy(stream);
  }
  void drop_graph() {
    if (gexec) (void)hipGraphExecDestroy(gexec);
    if (graph) (void)hipGraphDestroy(graph);
    if (ar_gexec) (void)hipGraphExecDestroy(ar_gexec);
    if (ar_graph) (void)hipGraphDestroy(ar_graph);
    gexec = nullptr;
    graph = nullptr;
    ar_gexec = nullptr;
    ar_graph = nullptr;
  }
  // Captures body() (which enqueues on `stream`) into a graph once; later calls reuse it.
  template <class F>
  int capture_once(hipGraph_t& g_out, hipGraphExec_t& ge, F&& body) {
    if (ge) return RT_OK;
    HIPCHK(hipStreamBeginCapture(stream, hipStreamCaptureModeThreadLocal));
    int st = body();
    hipGraph_t g = nullptr;
    hipError_t ce = hipStreamEndCapture(stream, &g);
    if (st != RT_OK) { if (g) (void)hipGraphDestroy(g); return st; }
    if (ce != hipSuccess) return fail(RT_ERR_HIP, "graph capture: %s", hipGetErrorString(ce));
    g_out = g;
    HIPCHK(hipGraphInstantiate(&ge, g_out, nullptr, nullptr, 0));
    return RT_OK;
  }
  template <class X> X* at(size_t off) const { return reinterpret_cast<X*>(ws + off); }
  virtual int init(const void* const* w) = 0;
  virtual int prefill(int ns, const int32_t* lens, const int32_t* ids, int budget, int32_t* first) = 0;
  virtual int run_round(bool forced) = 0;
  virtual int run_ar_step() = 0;
  int round(const int32_t* forced, int32_t* tokens, int32_t* n_comm, int32_t* acc);
  int round_static(int32_t* d_tokens, int32_t* d_n_comm, int32_t* d_acc);
  int ar_steps(int n, int32_t* tokens, int32_t* n_gen);
  int profile_round(rt_kernel_stat* stats, double* stage_ms, int32_t* tokens, int32_t* n_comm, int32_t* acc);
  int time_kernel(int kind, int reps, rt_kernel_stat* out);
  int debug_read(int id, int seq, void* dst, size_t bytes, size_t pos0 = 0);
  int trace_read(int id, int seq, void* dst, size_t bytes);
  int debug_write(int id, int seq, const void* src, size_t bytes);
};

template <typename T, typename K>
struct Engine : EngineBase {
  const char* tlayer(int l) const { return ws + p.t_layers + (size_t)l * p.layer_bytes; }
  const char* dlayer(int l) const { return ws + p.d_layers + (size_t)l * p.layer_bytes; }

  // Algorithmic bytes an epilogue moves for an M x N result (outputs written, side
  // inputs read).
  static double epi_bytes(const EpiArgs& e, int M, int N, int slabs) {
    const double mn = (double)M * N;
    switch (e.kind) {
      case EPI_STORE_F32: return mn * 4;
      case EPI_STORE_ACT: return mn * sizeof(T);
      case EPI_RESID: return mn * 8 + (e.cap ? mn * sizeof(T) : 0);
      case EPI_SWIGLU: return mn / 2 * sizeof(T);
      case EPI_COND_R: return mn * 8;
      case EPI_COND_GATE: return mn * 4;
      case EPI_PARTIAL: return mn * 4 * slabs;
      default: return mn * (12 + sizeof(T));   // EPI_COND_OUT: gate, e rows, x and etilde
    }
  }

  int gemm_call(int kind, const void* A, int lda, int a_rows, bool af32, const void* B, int N, int Kp, int M,
                EpiArgs e, int k_logical = 0, int partial_slabs = kResidSplits) {
    if (M <= 0) return RT_OK;
    if (k_logical <= 0) k_logical = Kp;
    e.M = M;
    e.N = N;
    // skinny up to 32 rows, and up to 64 rows with bf16 operands; the test hook (flags & 4)
    // keeps 33..64 rows on the wide split-k path
    const bool skinny = M <= 32 || (M <= 64 && sizeof(T) == 2 && !af32 && !(flags & 4));
    const int shape = skinny ? SHAPE_SKINNY : SHAPE_WIDE;
    const int KT = Kp / 32;
    int ks = 1;
    // bf16 GEMMs of 33..512 rows go to the mid-size kernel (which picks its own k slabs);
    // the test hook (flags & 4) keeps them on the 128x128 split-k path instead
    const bool mid = shape == SHAPE_WIDE && sizeof(T) == 2 && M <= 512 && !(flags & 4);
    if (shape == SHAPE_WIDE && !mid) {
      const int tiles = ((N + 127) / 128) * ((M + 127) / 128);
      if (flags & 4) {                       // test hook: force a k split wherever possible
        ks = KT < 4 ? KT : 4;
      } else if (tiles < 256) {
        ks = (320 + tiles - 1) / tiles;
        int maxk = KT / 4;
        if (maxk < 1) maxk = 1;
        if (ks > maxk) ks = maxk;
      }
      while (ks > 1 && (size_t)tiles * ks * 128 * 128 > kPartialFloats) --ks;
      if (tiles > kMaxTiles) ks = 1;
    }
    if (e.kind == EPI_PARTIAL) ks = partial_slabs;
    GemmArgs a;
    a.A = A; a.lda = lda; a.a_rows = a_rows; a.B = B; a.Kp = Kp; a.ksplit = ks;
    a.partial = pat<float>(p.partial, p.s_partial); a.counters = pat<uint32_t>(p.counters, p.s_counters);
    a.partial_floats = kPartialFloats;
    a.e = e;
    if (instrumented()) {
      const double Kl = (double)k_logical;
      prof_begin(kind, (double)N * Kl * sizeof(T) + (double)M * Kl * (af32 ? 4 : sizeof(T)) + epi_bytes(e, M, N, e.kind == EPI_PARTIAL ? ks : 1),
                 2.0 * M * N * Kl);
    }
    HIPCHK(gemm<T>(a, shape, af32, stream));
    prof_end();
    return RT_OK;
  }

  // k slabs of the q|k|v projection of M rows when it runs on the mid-size kernel
  // (bf16, 65..512 rows; the test hook keeps the wide path), else 1
  int qkv_slabs(int M) const {
    if (sizeof(T) != 2 || (flags & 4) || M <= 64 || M > 512) return 1;
    GemmArgs g{};
    g.Kp = p.Kp_d; g.partial_floats = kPartialFloats;
    g.e.kind = EPI_STORE_F32; g.e.M = M; g.e.N = p.qkvN;
    return gemm_mid_store_slabs(g, false);
  }

  struct LayerCtx {
    int M, rows_per_seq, n_seqs, stride, causal, splits, rb, rb_rows;
    const int32_t* pos0;
    const int32_t* nq;
    const int32_t* pt;
    T* kc;
    T* vc;
    T* cap;                      // packed capture buffer of the updated residual (null: none)
    int cap_k0;                  // column offset of this layer's slot in the capture
    const int32_t* prof_ctx;     // host copy of each sequence's context length (profiling only)
    int defer;                   // o / down (<= 32 rows): k-slab partials, added by the next norm
    int trace = -1;              // layer-trace record of this layer (-1: none)
  };
  // partials of the last deferred residual GEMM, consumed by the next norm of x
  NormFold pend{};
  // RMSNorm of x (rows of the residual stream) into the packed xa operand, folding in
  // any deferred residual partials first
  void norm_x(const T* w, int rows, K* keep, int ldk) {
    const Plan& q = p;
    prof_begin(RT_K_NORM, (double)rows * q.d * (4 + sizeof(T) + (keep ? q.ksz : 0)) +
                              (pend.n_part ? (double)rows * q.d * 4 * (pend.n_part + 1) : 0.0), 0);
    rmsnorm<T, K>(at<float>(q.x), q.d, w, q.d, cfg.rms_eps, rows, at<T>(q.xa), 16 * q.Kp_d, keep, ldk, pend, stream);
    prof_end();
    pend = NormFold{};
  }
  // o / down projection with the residual add, deferred (k slabs) or in the epilogue
  int resid_gemm(int kind, const LayerCtx& c, const void* A, int lda, const char* W, int Kp, int k_logical,
                 bool capture) {
    const Plan& q = p;
    EpiArgs e{};
    if (c.defer && c.M <= q.rpart_rows && (c.M <= 32 || (sizeof(T) == 2 && !(flags & 4)))) {
      const size_t stride = (size_t)q.rpart_rows * q.d;
      // skinny rows: 4 slabs; 65..512 rows (mid-size kernel): the slab count that fills
      // the chip (e.g. 40 column tiles x 6 slabs at the 14B shape), at most 8
      int ks = kResidSplits;
      if (c.M > 64 && sizeof(T) == 2) {
        GemmArgs g{};
        g.Kp = Kp; g.partial_floats = (size_t)kResidSplitsMax * stride;
        g.e.kind = EPI_PARTIAL; g.e.M = c.M; g.e.N = q.d;
        ks = gemm_mid_partial_slabs(g, false, kResidSplitsMax);
      }
      e.kind = EPI_PARTIAL; e.out_f32 = pat<float>(q.rpart, q.s_rpart); e.ldo = q.d; e.part_stride = stride;
      CHK(gemm_call(kind, A, lda, q.Mrows, false, W, q.d, Kp, c.M, e, k_logical, ks));
      pend = NormFold{pat<float>(q.rpart, q.s_rpart), ks, stride, capture ? (void*)c.cap : nullptr, 16 * q.Kp_nc,
                      c.cap_k0};
      return RT_OK;
    }
    e.kind = EPI_RESID; e.resid = at<float>(q.x); e.ldr = q.d;
    if (capture) { e.cap = c.cap; e.ldcap = 16 * q.Kp_nc; e.cap_k0 = c.cap_k0; }
    return gemm_call(kind, A, lda, q.Mrows, false, W, q.d, Kp, c.M, e, k_logical);
  }

  int layer(const char* lw, const LayerCtx& c) {
    const Plan& q = p;
    float* x = at<float>(q.x);
    T* xa = at<T>(q.xa);
    norm_x((const T*)(lw + q.lo_in), c.M, nullptr, 0);
    CHK(trace_item(c.trace, TI_X, x));   // the norm has folded any deferred partials into x
    // q|k|v on the mid-size kernel with k slabs: the slabs go to the split buffer and
    // qkv_post adds them (in slab order, as the slab epilogue would) while reading
    const int qks = qkv_slabs(c.M);
    EpiArgs e{};
    if (qks > 1) {
      e.kind = EPI_PARTIAL; e.out_f32 = pat<float>(q.partial, q.s_partial); e.ldo = q.qkvN;
      e.part_stride = (size_t)c.M * q.qkvN;
    } else {
      e.kind = EPI_STORE_F32; e.out_f32 = at<float>(q.qkvf); e.ldo = q.qkvN;
    }
    CHK(gemm_call(RT_K_GEMM_QKV, xa, 16 * q.Kp_d, q.Mrows, false, lw + q.lo_qkv, q.qkvN, q.Kp_d, c.M, e, q.d, qks));
    // Rounds and target-only steps (at most 16 rows per sequence, bf16, one q|k|v slab):
    // the attention kernel does the q / k-norm, the rotation and the block's K / V cache
    // write itself (debug flag 16 keeps the separate kernel)
    const bool fusable = sizeof(T) == 2 && qks == 1 && c.nq == nullptr && c.rows_per_seq <= 16 &&
                         (q.hd == 64 || q.hd == 128);
    const bool fuse = fusable && !(flags & 16);
    if (!fuse) {
      QkvPostArgs qp{};
      qp.src = qks > 1 ? pat<float>(q.partial, q.s_partial) : at<float>(q.qkvf); qp.lds = q.qkvN; qp.M = c.M;
      qp.n_part = qks; qp.part_stride = (size_t)c.M * q.qkvN;
      qp.q_cols = q.qN; qp.kv_cols = q.kvN; qp.layer_cols = q.qkvN; qp.n_layers = 1;
      qp.head_dim = q.hd; qp.n_kv_heads = q.Hkv; qp.q_out = at<T>(q.qbuf); qp.ldq = q.qN;
      qp.q_norm = lw + q.lo_qn; qp.k_norm = lw + q.lo_kn; qp.norm_layer_stride = 0;
      qp.kcache = c.kc; qp.vcache = c.vc; qp.cache_layer_stride = 0;
      qp.page_table = c.pt; qp.max_pages = q.pages_per_seq;
      qp.rope = at<float>(q.rope); qp.rope_max_pos = q.T; qp.eps = cfg.rms_eps;
      qp.rows_per_seq = c.rows_per_seq; qp.seq_stride = c.stride; qp.pos0 = c.pos0; qp.nrows = nullptr;
      prof_begin(RT_K_QKV_POST, (double)c.M * q.qkvN * (4 * qks + sizeof(T)), 0);
      HIPCHK(qkv_post<T>(qp, stream));
      prof_end();
      CHK(trace_item(c.trace, TI_Q, at<T>(q.qbuf)));
    }
    AttnArgs a{};
    a.q = at<T>(q.qbuf); a.kcache = c.kc; a.vcache = c.vc; a.page_table = c.pt; a.max_pages = q.pages_per_seq;
    a.pos0 = c.pos0; a.nq = c.nq; a.seq_stride = c.stride; a.rows_per_seq = c.rows_per_seq;
    a.n_seqs = c.n_seqs; a.causal = c.causal; a.n_q_heads = q.Hq; a.n_kv_heads = q.Hkv; a.head_dim = q.hd;
    a.splits = c.splits; a.row_blocks = c.rb; a.rb_rows = c.rb_rows;
    // batches whose attention never takes the q / k work (so the fused and separate forms,
    // compared by a test hook, share one plan) may span unit boundaries
    a.span = fusable ? 0 : (flags & 64) ? 2 : 1;
    a.opart = pat<float>(q.opart, q.s_opart); a.mlpart = pat<float>(q.mlpart, q.s_mlpart);
    a.plan = pat<int32_t>(q.attn_plan, q.s_attn_plan);
    a.out = at<T>(q.attn); a.ldo = 16 * q.Kp_q; a.scale = 1.0f / sqrtf((float)q.hd);
    if (fuse) {
      a.qkv = at<float>(q.qkvf); a.ldqkv = q.qkvN; a.q_cols = q.qN; a.kv_cols = q.kvN;
      a.q_norm = lw + q.lo_qn; a.k_norm = lw + q.lo_kn;
      a.rope = at<float>(q.rope); a.rope_max_pos = q.T; a.eps = cfg.rms_eps;
      a.q_out = c.trace >= 0 ? at<T>(q.qbuf) : nullptr; a.ldq = q.qN;
    }
    if (instrumented()) {
      // keys read: every sequence's context plus the block, K and V, once per KV head;
      // fused: the fp32 q|k|v rows read and the block's K / V written instead of bf16 q
      double keys = 0;
      for (int s = 0; s < c.n_seqs; ++s) keys += (double)(c.prof_ctx[s] + c.rows_per_seq);
      const double kvb = keys * 2.0 * q.Hkv * q.hd * sizeof(T);
      const double rows = (double)c.n_seqs * c.rows_per_seq;
      const double qio = fuse ? rows * (q.qkvN * 4.0 + 2.0 * q.kvN * sizeof(T)) : rows * q.qN * sizeof(T);
      prof_begin(RT_K_ATTENTION, kvb + qio + rows * q.qN * sizeof(T), 4.0 * keys * c.rows_per_seq * q.Hq * q.hd);
    }
    HIPCHK(attention_partials<T>(a, stream));
    prof_end();
    if (a.splits > 1) {
      // partials: unnormalised O plus (max, sum) per (row, split), read once
      prof_begin(RT_K_ATTN_MERGE, (double)a.splits * q.Hkv * c.rb * c.n_seqs * c.rb_rows * (q.hd + 2) * 4.0, 0);
      HIPCHK(attention_merge<T>(a, stream));
      prof_end();
    }
    if (fuse) CHK(trace_item(c.trace, TI_Q, at<T>(q.qbuf)));
    CHK(trace_item(c.trace, TI_ATTN, at<T>(q.attn)));
    CHK(resid_gemm(RT_K_GEMM_O, c, at<T>(q.attn), 16 * q.Kp_q, lw + q.lo_o, q.Kp_q, q.qN, false));
    norm_x((const T*)(lw + q.lo_post), c.M, nullptr, 0);
    CHK(trace_item(c.trace, TI_XMID, x));
    CHK(trace_item(c.trace, TI_H2, xa));
    e = EpiArgs{};
    e.kind = EPI_SWIGLU; e.out_act = at<T>(q.mlp); e.ldo = 16 * q.Kp_F;
    CHK(gemm_call(RT_K_GEMM_GATE_UP, xa, 16 * q.Kp_d, q.Mrows, false, lw + q.lo_gu, 2 * q.F, q.Kp_d, c.M, e, q.d));
    CHK(trace_item(c.trace, TI_MLP, at<T>(q.mlp)));
    CHK(resid_gemm(RT_K_GEMM_DOWN, c, at<T>(q.mlp), 16 * q.Kp_F, lw + q.lo_down, q.Kp_F, q.F, c.cap != nullptr));
    return RT_OK;
  }

  // LM head over rows of xa with a fused argmax into keys[M] (optional fp32 logits).
  int lm_head_argmax(int M, uint64_t* keys, float* logits) {
    const Plan& q = p;
    if (sizeof(T) == 2 && M > 32 && M <= 512) {   // mid-size rows: one pass over the vocabulary
      GemmArgs g{};
      g.A = at<T>(q.xa); g.lda = 16 * q.Kp_d; g.a_rows = q.Mrows; g.B = at<T>(q.lm_head); g.Kp = q.Kp_d; g.ksplit = 1;
      g.e.kind = EPI_ARGMAX; g.e.M = M; g.e.N = q.V; g.e.out_f32 = logits; g.e.ldo = q.V;
      g.e.part_keys = at<uint64_t>(q.part_keys);
      const int parts = 2 * ((q.V + gemm_mid_cols(q.V, M) - 1) / gemm_mid_cols(q.V, M));
      prof_begin(RT_K_LM_HEAD, (double)q.V * q.d * sizeof(T) + (double)M * q.d * sizeof(T), 2.0 * M * q.V * q.d);
      g.partial = pat<float>(q.partial, q.s_partial); g.partial_floats = kPartialFloats;
      HIPCHK(gemm_mid(g, false, stream));
      prof_end();
      prof_begin(RT_K_MISC, (double)parts * M * 8, 0);
      HIPCHK(argmax_reduce(at<uint64_t>(q.part_keys), parts, M, keys, stream));
      prof_end();
      return RT_OK;
    }
    for (int r0 = 0; r0 < M; r0 += 32) {          // 32-row passes over the vocabulary
      const int m = M - r0 < 32 ? M - r0 : 32;
      const int parts = lmhead_parts(m, q.V, q.Kp_d, (int)sizeof(T));
      LmHeadArgs h{};
      h.A = at<T>(q.xa) + (size_t)(r0 / 16) * 16 * q.Kp_d; h.lda = 16 * q.Kp_d; h.a_rows = q.Mrows - r0; h.M = m;
      h.B = at<T>(q.lm_head); h.N = q.V; h.Kp = q.Kp_d;
      h.part_keys = at<uint64_t>(q.part_keys); h.logits = logits ? logits + (size_t)r0 * q.V : nullptr;
      h.ldl = q.V;
      prof_begin(RT_K_LM_HEAD, (double)q.V * q.d * sizeof(T) + (double)m * q.d * sizeof(T), 2.0 * m * q.V * q.d);
      HIPCHK(lm_head<T>(h, stream));
      prof_end();
      prof_begin(RT_K_MISC, (double)parts * m * 8, 0);
      HIPCHK(argmax_reduce(at<uint64_t>(q.part_keys), parts, m, keys + r0, stream));
      prof_end();
    }
    return RT_OK;
  }

  bool sampling() const { return cfg.temperature > 0.f; }
  // Filtered distributions of `rows` rows of fp32 logits (and, per mode, one draw per row).
  int dists(const float* logits, int rows, int32_t* ids, float* probs, int mode, int seq0, int32_t* tok_out) {
    const Plan& q = p;
    DistArgs d{};
    d.logits = logits; d.ldl = q.V; d.V = q.V; d.rows = rows;
    d.top_k = cfg.top_k; d.inv_temp = 1.0f / cfg.temperature; d.top_p = cfg.top_p;
    d.ids = ids; d.probs = probs; d.ldd = kMaxTopK;
    d.mode = mode; d.state = at<int32_t>(q.state); d.state_stride = kStateFields; d.bk = q.bk; d.seq0 = seq0;
    d.seed = cfg.sample_seed; d.tok_out = tok_out;
    prof_begin(RT_K_MISC, (double)rows * q.V * 4 * 4, 0);
    HIPCHK(filtered_dists(d, at<uint64_t>(q.topk_cand), stream));
    prof_end();
    return RT_OK;
  }

  int cond_slot(int l) const {
    for (int i = 0; i < cfg.n_cond_layers; ++i)
      if (cfg.cond_layer_ids[i] == l) return i;
    return -1;
  }

  // Drafter context pathway for M rows: fc -> RMSNorm -> per-layer K (k-norm, RoPE) / V.
  int context_append(int M, int rows_per_seq, const int32_t* pos0, const int32_t* nrows, int stride,
                     const int32_t* pt) {
    const Plan& q = p;
    EpiArgs e{};
    e.kind = EPI_STORE_F32; e.out_f32 = at<float>(q.fcout); e.ldo = q.d;
    CHK(gemm_call(RT_K_GEMM_CONTEXT, at<T>(q.g), 16 * q.Kp_nc, q.Mrows, false, at<T>(q.fc), q.d, q.Kp_nc, M, e, q.nc * q.d));
    prof_begin(RT_K_NORM, (double)M * q.d * (4 + sizeof(T)), 0);
    rmsnorm<T, K>(at<float>(q.fcout), q.d, at<T>(q.hidden_norm), q.d, cfg.rms_eps, M, at<T>(q.fa), 16 * q.Kp_d,
                  nullptr, 0, NormFold{}, stream);
    prof_end();
    e = EpiArgs{};
    e.kind = EPI_STORE_F32; e.out_f32 = at<float>(q.qkvf); e.ldo = q.LD * 2 * q.kvN;
    CHK(gemm_call(RT_K_GEMM_CONTEXT, at<T>(q.fa), 16 * q.Kp_d, q.Mrows, false, at<T>(q.ctxkv), q.LD * 2 * q.kvN, q.Kp_d, M, e, q.d));
    QkvPostArgs qp{};
    qp.src = at<float>(q.qkvf); qp.lds = q.LD * 2 * q.kvN; qp.M = M;
    qp.q_cols = 0; qp.kv_cols = q.kvN; qp.layer_cols = 2 * q.kvN; qp.n_layers = q.LD;
    qp.head_dim = q.hd; qp.n_kv_heads = q.Hkv;
    qp.k_norm = at<T>(q.ctx_knorm); qp.norm_layer_stride = q.hd;
    qp.kcache = at<T>(q.dkc); qp.vcache = at<T>(q.dvc); qp.cache_layer_stride = q.cache_layer_elems;
    qp.page_table = pt; qp.max_pages = q.pages_per_seq;
    qp.rope = at<float>(q.rope); qp.rope_max_pos = q.T; qp.eps = cfg.rms_eps;
    qp.rows_per_seq = rows_per_seq; qp.seq_stride = stride; qp.pos0 = pos0; qp.nrows = nrows;
    prof_begin(RT_K_QKV_POST, (double)M * q.LD * 2 * q.kvN * (4 + sizeof(T)), 0);
    HIPCHK(qkv_post<T>(qp, stream));
    prof_end();
    return RT_OK;
  }

  int init(const void* const* w) override {
    const Plan& q = p;
    const size_t E = sizeof(T);
    auto W = [&](int i) { return (const T*)w[i]; };
    auto copy = [&](size_t off, int i, size_t n) {
      return hipMemcpyAsync(ws + off, w[i], n * E, hipMemcpyDeviceToDevice, stream);
    };
    fill_zero(ws + q.zero_from, q.total - q.zero_from, stream);
    HIPCHK(hipGetLastError());
    HIPCHK(copy(q.embed, 0, (size_t)q.V * q.d));
    auto pack_layer = [&](char* base, int widx) -> int {
      T* qkv = (T*)(base + q.lo_qkv);
      pack_weights<T>(W(widx + 1), q.qN, q.d, q.Kp_d, qkv, stream);
      pack_weights<T>(W(widx + 2), q.kvN, q.d, q.Kp_d, qkv + (size_t)q.qN * q.Kp_d, stream);
      pack_weights<T>(W(widx + 3), q.kvN, q.d, q.Kp_d, qkv + (size_t)(q.qN + q.kvN) * q.Kp_d, stream);
      pack_weights<T>(W(widx + 6), q.d, q.qN, q.Kp_q, (T*)(base + q.lo_o), stream);
      pack_interleaved<T>(W(widx + 8), W(widx + 9), q.F, q.d, q.Kp_d, (T*)(base + q.lo_gu), stream);
      pack_weights<T>(W(widx + 10), q.d, q.F, q.Kp_F, (T*)(base + q.lo_down), stream);
      HIPCHK(hipMemcpyAsync(base + q.lo_in, w[widx + 0], q.d * E, hipMemcpyDeviceToDevice, stream));
      HIPCHK(hipMemcpyAsync(base + q.lo_post, w[widx + 7], q.d * E, hipMemcpyDeviceToDevice, stream));
      HIPCHK(hipMemcpyAsync(base + q.lo_qn, w[widx + 4], q.hd * E, hipMemcpyDeviceToDevice, stream));
      HIPCHK(hipMemcpyAsync(base + q.lo_kn, w[widx + 5], q.hd * E, hipMemcpyDeviceToDevice, stream));
      HIPCHK(hipGetLastError());
      return RT_OK;
    };
    for (int l = 0; l < q.L; ++l) CHK(pack_layer(ws + q.t_layers + (size_t)l * q.layer_bytes, 1 + 11 * l));
    const int b2 = 1 + 11 * q.L;
    HIPCHK(copy(q.t_final_norm, b2, q.d));
    pack_weights<T>(W(b2 + 1), q.V, q.d, q.Kp_d, at<T>(q.lm_head), stream);
    pack_weights<T>(W(b2 + 2), q.d, q.nc * q.d, q.Kp_nc, at<T>(q.fc), stream);
    HIPCHK(copy(q.hidden_norm, b2 + 3, q.d));
    for (int l = 0; l < q.LD; ++l) {
      const int widx = b2 + 4 + 11 * l;
      CHK(pack_layer(ws + q.d_layers + (size_t)l * q.layer_bytes, widx));
      T* ck = at<T>(q.ctxkv) + (size_t)2 * l * q.kvN * q.Kp_d;
      pack_weights<T>(W(widx + 2), q.kvN, q.d, q.Kp_d, ck, stream);
      pack_weights<T>(W(widx + 3), q.kvN, q.d, q.Kp_d, ck + (size_t)q.kvN * q.Kp_d, stream);
      HIPCHK(hipMemcpyAsync(at<T>(q.ctx_knorm) + (size_t)l * q.hd, w[widx + 5], q.hd * E,
                            hipMemcpyDeviceToDevice, stream));
    }
    const int b3 = b2 + 4 + 11 * q.LD;
    HIPCHK(copy(q.d_final_norm, b3, q.d));
    pack_weights<T>(W(b3 + 1), q.d, 2 * q.d, q.Kp_2d, at<T>(q.wc), stream);
    pack_weights<T>(W(b3 + 2), q.d, q.d, q.Kp_d, at<T>(q.wv), stream);
    pack_weights<T>(W(b3 + 3), q.d, 2 * q.d, q.Kp_2d, at<T>(q.wg), stream);
    if (cfg.cond_mode == RT_COND_LOWRANK) {
      // [A | 0] (A acts on m only) above C_down, as one packed [96][2d] matrix
      pack_weights<T>(W(b3 + 4), kLowRankLatent, q.d, q.Kp_2d, at<T>(q.lr_down), stream);
      pack_weights<T>(W(b3 + 5), kLowRankCorr, 2 * q.d, q.Kp_2d, at<T>(q.lr_down) + (size_t)kLowRankLatent * q.Kp_2d,
                      stream);
      HIPCHK(copy(q.lr_cup, b3 + 6, (size_t)kLowRankLatent * kLowRankCorr));
      HIPCHK(copy(q.lr_v, b3 + 7, (size_t)q.d * kLowRankLatent));
      HIPCHK(copy(q.lr_g, b3 + 8, (size_t)q.d * kLowRankLatent));
      lowrank_gate_bias<T>(W(b3 + 3), at<T>(q.embed), q.d, cfg.mask_token_id, at<float>(q.lr_ge), stream);
    }
    HIPCHK(hipGetLastError());
    // page table: page j of sequence s is pool page j * max_batch + s
    std::vector<int32_t> pt((size_t)q.n_pages);
    for (int s = 0; s < q.bmax; ++s)
      for (int j = 0; j < q.pages_per_seq; ++j) pt[(size_t)s * q.pages_per_seq + j] = j * q.bmax + s;
    HIPCHK(hipMemcpyAsync(ws + q.page_table, pt.data(), pt.size() * 4, hipMemcpyHostToDevice, stream));
    // RoPE table: angle = fp32(pos * fp32(theta^(-2i/hd))); cos and sin rounded to fp32
    const int half = q.hd / 2;
    std::vector<float> rope((size_t)q.T * half * 2);
    for (int i = 0; i < half; ++i) {
      const float inv = (float)pow((double)cfg.rope_theta, -2.0 * i / q.hd);
      for (int pos = 0; pos < q.T; ++pos) {
        const float ang = (float)pos * inv;
        rope[(size_t)pos * half + i] = (float)cos((double)ang);
        rope[(size_t)q.T * half + (size_t)pos * half + i] = (float)sin((double)ang);
      }
    }
    HIPCHK(hipMemcpyAsync(ws + q.rope, rope.data(), rope.size() * 4, hipMemcpyHostToDevice, stream));
    HIPCHK(hipStreamSynchronize(stream));
    return RT_OK;
  }

  int prefill(int ns, const int32_t* lens, const int32_t* ids, int budget, int32_t* first) override {
    const Plan& q = p;
    drop_graph();
    prefilled = false;
    ar_mode = false;
    size_t off = 0;
    int32_t* pf = at<int32_t>(q.pf_ints);
    int32_t* tok = at<int32_t>(q.tokbuf);
    for (int s = 0; s < ns; ++s) {
      const int len = lens[s];
      HIPCHK(hipMemcpyAsync(tok, ids + off, (size_t)len * 4, hipMemcpyHostToDevice, stream));
      const int32_t* pt = at<int32_t>(q.page_table) + (size_t)s * q.pages_per_seq;
      for (int c0 = 0; c0 < len; c0 += q.PF) {
        const int n = len - c0 < q.PF ? len - c0 : q.PF;
        set_ints(pf, 2, c0, n, 0, 0, stream);
        embed_rows<T>(at<T>(q.embed), q.d, tok + c0, n, at<float>(q.x), q.d, stream);
        for (int l = 0; l < q.L; ++l) {
          const int slot = cond_slot(l);
          LayerCtx c{n, q.PF, 1, 0, 1, 1, (n * q.G + kAttnRows - 1) / kAttnRows, kAttnRows, pf, pf + 1, pt,
                     at<T>(q.kc) + (size_t)l * q.cache_layer_elems, at<T>(q.vc) + (size_t)l * q.cache_layer_elems,
                     slot >= 0 ? at<T>(q.g) : nullptr, slot * q.d, &c0};
          CHK(layer(tlayer(l), c));
        }
        CHK(context_append(n, q.PF, pf, nullptr, 0, pt));
        if (c0 + n == len) {
          rmsnorm<T, K>(at<float>(q.x) + (size_t)(n - 1) * q.d, q.d, at<T>(q.t_final_norm), q.d, cfg.rms_eps, 1,
                        at<T>(q.xa), 16 * q.Kp_d, nullptr, 0, NormFold{}, stream);
          const bool smp = sampling();
          CHK(lm_head_argmax(1, at<uint64_t>(q.tkeys), smp ? at<float>(q.vlogits) : nullptr));
          if (smp)
            CHK(dists(at<float>(q.vlogits), 1, at<int32_t>(q.dist_ids_v), at<float>(q.dist_p_v), SAMPLE_FIRST, s,
                      at<int32_t>(q.stok)));
          first_token(at<int32_t>(q.state), s, at<uint64_t>(q.tkeys), smp ? at<int32_t>(q.stok) : nullptr, len, budget,
                      at<int32_t>(q.first_tok), stream);
        }
        HIPCHK(hipGetLastError());
      }
      HIPCHK(hipStreamSynchronize(stream));   // the token buffer is reused by the next sequence
      off += (size_t)len;
    }
    fill_zero(ws + q.hd_keep, (size_t)q.R * q.d * q.ksz, stream);
    fill_zero(ws + q.ht_keep, (size_t)q.R * q.d * q.ksz, stream);
    HIPCHK(hipMemcpyAsync(h_out, ws + q.first_tok, (size_t)ns * 4, hipMemcpyDeviceToHost, stream));
    HIPCHK(hipStreamSynchronize(stream));
    memcpy(first, h_out, (size_t)ns * 4);
    n_seqs = ns;
    prefilled = true;
    return RT_OK;
  }

  int run_round(bool forced) override {
    const Plan& q = p;
    const int R = n_seqs * q.bk;
    int32_t* st = at<int32_t>(q.state);
    float* x = at<float>(q.x);
    T* xa = at<T>(q.xa);
    const int32_t* pt = at<int32_t>(q.page_table);
    // (1) rejected-trajectory conditioning (Eq.5-9)
    stage(0);
    if (cfg.cond_mode == RT_COND_RETRACE || cfg.cond_mode == RT_COND_RAW_GATED) {
      const bool raw = cfg.cond_mode == RT_COND_RAW_GATED;
      prof_begin(RT_K_MISC, (double)R * q.d * ((raw ? 2 : 4) * q.ksz + sizeof(T) + (raw ? 8 : 16)), 0);
      const int ldg2 = 16 * q.Kp_2d;
      cond_prep<T, K>(at<T>(q.embed), q.d, st, cfg.mask_token_id, at<K>(q.hd_keep), at<K>(q.ht_keep), n_seqs, q.bk,
                      at<float>(q.mu), at<float>(q.er), ldg2, raw ? 1 : 0, stream);
      prof_end();
      EpiArgs e{};
      if (!raw) {   // corrected signal r = m + beta W_c [m; u] (Eq.7-8); raw gated keeps r = m
        e.kind = EPI_COND_R; e.out_f32 = at<float>(q.er); e.ldo = ldg2; e.out_k0 = q.d;
        e.cond_m = at<float>(q.mu); e.ld_cond_m = ldg2; e.beta = cfg.beta;
        CHK(gemm_call(RT_K_GEMM_COND, at<float>(q.mu), ldg2, R, true, at<T>(q.wc), q.d, q.Kp_2d, R, e, 2 * q.d));
        e = EpiArgs{};
      }
      e.kind = EPI_COND_GATE; e.out_f32 = at<float>(q.gate); e.ldo = q.d;
      CHK(gemm_call(RT_K_GEMM_COND, at<float>(q.er), ldg2, R, true, at<T>(q.wg), q.d, q.Kp_2d, R, e, 2 * q.d));
      e = EpiArgs{};
      e.kind = EPI_COND_OUT; e.resid = x; e.ldr = q.d; e.etilde = at<float>(q.etilde);
      e.gate = at<float>(q.gate); e.ld_gate = q.d; e.embed = at<T>(q.embed); e.mask_token = cfg.mask_token_id;
      e.anchor = st + ST_ANCHOR; e.cond_len = st + ST_COND_LEN; e.seq_stride = kStateFields;
      e.rows_per_seq = q.bk;
      // r occupies packed k tiles d/32 .. 2d/32 of er
      CHK(gemm_call(RT_K_GEMM_COND, at<float>(q.er) + (size_t)(q.d / 32) * 512, ldg2, R, true, at<T>(q.wv), q.d, q.Kp_d, R, e, q.d));
    } else if (cfg.cond_mode == RT_COND_LOWRANK) {
      prof_begin(RT_K_MISC, (double)R * q.d * (4 * q.ksz + sizeof(T) + 16), 0);
      const int ldg2 = 16 * q.Kp_2d;
      cond_prep<T, K>(at<T>(q.embed), q.d, st, cfg.mask_token_id, at<K>(q.hd_keep), at<K>(q.ht_keep), n_seqs, q.bk,
                      at<float>(q.mu), at<float>(q.er), ldg2, 0, stream);
      prof_end();
      EpiArgs e{};
      e.kind = EPI_STORE_F32; e.out_f32 = at<float>(q.lr_lat); e.ldo = kLowRankRows;
      CHK(gemm_call(RT_K_GEMM_COND, at<float>(q.mu), ldg2, R, true, at<T>(q.lr_down), kLowRankRows, q.Kp_2d, R, e,
                    2 * q.d));
      prof_begin(RT_K_MISC, (double)R * q.d * (sizeof(T) + 8) + (double)q.d * kLowRankLatent * 2 * sizeof(T), 0);
      lowrank_fuse<T>(at<float>(q.lr_lat), at<T>(q.lr_cup), at<T>(q.lr_v), at<T>(q.lr_g), at<float>(q.lr_ge), cfg.beta,
                      at<T>(q.embed), q.d, st, cfg.mask_token_id, n_seqs, q.bk, x, at<float>(q.etilde), stream);
      prof_end();
    } else {
      // plain block drafting, or the overwrite ablation (conditioned rows take m_j)
      const bool ow = cfg.cond_mode == RT_COND_OVERWRITE;
      prof_begin(RT_K_MISC, (double)R * q.d * (sizeof(T) + 8), 0);
      embed_block<T, K>(at<T>(q.embed), q.d, st, cfg.mask_token_id, n_seqs, q.bk, ow ? at<K>(q.hd_keep) : nullptr,
                        x, at<float>(q.etilde), q.d, stream);
      prof_end();
    }
    stage(1);
    // (2) drafter: B+1 rows at P..P+B over its context cache (no causal mask in the block)
    for (int l = 0; l < q.LD; ++l) {
      LayerCtx c{R, q.bk, n_seqs, kStateFields, 0, q.attn_splits, q.attn_rb, q.attn_rows, st + ST_SEQ_LEN, nullptr, pt,
                 at<T>(q.dkc) + (size_t)l * q.cache_layer_elems, at<T>(q.dvc) + (size_t)l * q.cache_layer_elems,
                 nullptr, 0, prof_ctx.data(), 1};
      c.trace = l;
      CHK(layer(dlayer(l), c));
    }
    stage(2);
    norm_x(at<T>(q.d_final_norm), R, at<K>(q.hd_keep), q.d);
    CHK(trace_item(q.LD + q.L, TI_X, x));
    CHK(trace_item(q.LD + q.L, TI_H2, xa));
    const bool smp = sampling();
    CHK(lm_head_argmax(R, at<uint64_t>(q.dkeys), (smp || (flags & 1)) ? at<float>(q.dlogits) : nullptr));
    // sampling: the drafter's filtered distributions, drafts drawn into dtok (unless forced)
    if (smp)
      CHK(dists(at<float>(q.dlogits), R, at<int32_t>(q.dist_ids_d), at<float>(q.dist_p_d), SAMPLE_DRAFT, 0,
                forced ? nullptr : at<int32_t>(q.dtok)));
    // (3) verify: [anchor, drafts] at P..P+B, causal over the target cache
    stage(3);
    prof_begin(RT_K_MISC, (double)R * q.d * (sizeof(T) + 4), 0);
    embed_verify<T>(at<T>(q.embed), q.d, st, at<uint64_t>(q.dkeys), (forced || smp) ? 1 : 0, at<int32_t>(q.dtok),
                    n_seqs, q.bk, x, q.d, stream);
    prof_end();
    for (int l = 0; l < q.L; ++l) {
      const int slot = cond_slot(l);
      LayerCtx c{R, q.bk, n_seqs, kStateFields, 1, q.attn_splits, q.attn_rb, q.attn_rows, st + ST_SEQ_LEN, nullptr, pt,
                 at<T>(q.kc) + (size_t)l * q.cache_layer_elems, at<T>(q.vc) + (size_t)l * q.cache_layer_elems,
                 slot >= 0 ? at<T>(q.g) : nullptr, slot * q.d, prof_ctx.data(), 1};
      c.trace = q.LD + l;
      CHK(layer(tlayer(l), c));
    }
    stage(4);
    norm_x(at<T>(q.t_final_norm), R, at<K>(q.ht_keep), q.d);
    CHK(trace_item(q.LD + q.L + 1, TI_X, x));
    CHK(trace_item(q.LD + q.L + 1, TI_H2, xa));
    CHK(lm_head_argmax(R, at<uint64_t>(q.tkeys), (smp || (flags & 1)) ? at<float>(q.vlogits) : nullptr));
    if (smp)
      CHK(dists(at<float>(q.vlogits), R, at<int32_t>(q.dist_ids_v), at<float>(q.dist_p_v), SAMPLE_NONE, 0, nullptr));
    // (4) acceptance, commit, rollback, carry / reset
    stage(5);
    prof_begin(RT_K_MISC, (double)R * 16, 0);
    if (smp) {
      AcceptSampleArgs g{};
      g.state = st; g.state_stride = kStateFields; g.dtok = at<int32_t>(q.dtok);
      g.q_ids = at<int32_t>(q.dist_ids_d); g.q_p = at<float>(q.dist_p_d);
      g.p_ids = at<int32_t>(q.dist_ids_v); g.p_p = at<float>(q.dist_p_v); g.ldd = kMaxTopK;
      g.tkeys = at<uint64_t>(q.tkeys); g.ttok = at<int32_t>(q.ttok); g.bk = q.bk; g.seed = cfg.sample_seed;
      g.out_tok = at<int32_t>(q.out_tok); g.out_n = at<int32_t>(q.out_n); g.out_a = at<int32_t>(q.out_a);
      HIPCHK(accept_sampled(g, n_seqs, stream));
    } else {
      accept(st, at<int32_t>(q.dtok), at<uint64_t>(q.tkeys), at<int32_t>(q.ttok), n_seqs, q.bk, at<int32_t>(q.out_tok),
             at<int32_t>(q.out_n), at<int32_t>(q.out_a), stream);
    }
    prof_end();
    // drafter context pathway for the committed rows 0..A at P..P+A
    stage(6);
    CHK(context_append(R, q.bk, st + ST_ROUND_POS, st + ST_APPEND, kStateFields, pt));
    stage(7);
    HIPCHK(hipGetLastError());
    return RT_OK;
  }

  // One target-only step (greedy or sampled): the anchor row of every sequence at position seq_len.
  int run_ar_step() override {
    const Plan& q = p;
    static_assert(kStateFields <= kStateSlots, "per-sequence state exceeds its slots");
    static_assert(kMaxTopK == RT_MAX_TOP_K, "distribution width");
    static_assert(kTopkChunk == kSelectChunk, "top-k stage size");
    static_assert(kLmGrid <= kLmPartsMin, "LM-head key rows");
    static_assert(kAttnRowsAr == kAttnRows, "target-only steps use the 64-row attention blocks");
    const int M = n_seqs;
    int32_t* st = at<int32_t>(q.state);
    const int32_t* pt = at<int32_t>(q.page_table);
    prof_begin(RT_K_MISC, (double)M * q.d * (sizeof(T) + 4), 0);
    embed_block<T, K>(at<T>(q.embed), q.d, st, cfg.mask_token_id, n_seqs, 1, nullptr, at<float>(q.x), nullptr,
                      q.d, stream);
    prof_end();
    for (int l = 0; l < q.L; ++l) {
      LayerCtx c{M, 1, n_seqs, kStateFields, 1, q.ar_splits, q.ar_rb, kAttnRows, st + ST_SEQ_LEN, nullptr, pt,
                 at<T>(q.kc) + (size_t)l * q.cache_layer_elems, at<T>(q.vc) + (size_t)l * q.cache_layer_elems,
                 nullptr, 0, prof_ctx.data(), 1};
      CHK(layer(tlayer(l), c));
    }
    norm_x(at<T>(q.t_final_norm), M, nullptr, 0);
    const bool smp = sampling();
    CHK(lm_head_argmax(M, at<uint64_t>(q.tkeys), (smp || (flags & 1)) ? at<float>(q.vlogits) : nullptr));
    if (smp)
      CHK(dists(at<float>(q.vlogits), M, at<int32_t>(q.dist_ids_v), at<float>(q.dist_p_v), SAMPLE_STEP, 0,
                at<int32_t>(q.stok)));
    prof_begin(RT_K_MISC, (double)M * 16, 0);
    ar_commit(st, at<uint64_t>(q.tkeys), smp ? at<int32_t>(q.stok) : nullptr, n_seqs, at<int32_t>(q.ar_tok),
              kArMaxSteps, at<int32_t>(q.pf_ints) + 8, stream);
    prof_end();
    HIPCHK(hipGetLastError());
    return RT_OK;
  }
};

static int ar_state_error() {
  return fail(RT_ERR_STATE, "target-only steps ran since rt_prefill (the drafter context was not extended); "
                            "call rt_prefill before the next round");
}

int EngineBase::ar_steps(int n, int32_t* tokens, int32_t* n_gen) {
  if (!prefilled) return fail(RT_ERR_STATE, "rt_ar_steps called before rt_prefill");
  if (!tokens || !n_gen) return fail(RT_ERR_INVALID, "null output pointer");
  if (n < 1 || n > kArMaxSteps) return fail(RT_ERR_INVALID, "n_steps must be in [1, %d]", kArMaxSteps);
  const Plan& q = p;
  ar_mode = true;
  set_ints(at<int32_t>(q.pf_ints) + 8, 1, 0, 0, 0, 0, stream);   // step counter (outside the graph)
  HIPCHK(hipGetLastError());
  if (flags & 2) {
    for (int i = 0; i < n; ++i) CHK(run_ar_step());
  } else {
    CHK(capture_once(ar_graph, ar_gexec, [&] { return run_ar_step(); }));
    for (int i = 0; i < n; ++i) HIPCHK(hipGraphLaunch(ar_gexec, stream));
  }
  std::vector<int32_t> h((size_t)n_seqs * kArMaxSteps);
  HIPCHK(hipMemcpyAsync(h.data(), ws + q.ar_tok, h.size() * 4, hipMemcpyDeviceToHost, stream));
  HIPCHK(hipStreamSynchronize(stream));
  for (int s = 0; s < n_seqs; ++s) {
    int cnt = 0;
    for (int i = 0; i < n; ++i) {
      const int32_t t = h[(size_t)s * kArMaxSteps + i];
      tokens[(size_t)s * n + i] = t;
      cnt += t >= 0;
    }
    n_gen[s] = cnt;
  }
  return RT_OK;
}

int EngineBase::round(const int32_t* forced, int32_t* tokens, int32_t* n_comm, int32_t* acc) {
  if (!prefilled) return fail(RT_ERR_STATE, "rt_spec_round called before rt_prefill");
  if (ar_mode) return ar_state_error();
  if (!tokens || !n_comm || !acc) return fail(RT_ERR_INVALID, "null output pointer");
  const Plan& q = p;
  if (forced) {
    std::vector<int32_t> h((size_t)n_seqs * q.bk, 0);
    for (int s = 0; s < n_seqs; ++s)
      for (int i = 1; i < q.bk; ++i) {
        const int32_t t = forced[(size_t)s * q.B + i - 1];
        if (t < 0 || t >= q.V) return fail(RT_ERR_TOKEN, "forced draft token %d out of range", t);
        h[(size_t)s * q.bk + i] = t;
      }
    HIPCHK(hipMemcpyAsync(ws + q.dtok, h.data(), h.size() * 4, hipMemcpyHostToDevice, stream));
    CHK(run_round(true));
  } else if (flags & 10) {   // eager launches (debug flag 2, or the layer trace)
    CHK(run_round(false));
  } else {
    CHK(capture_once(graph, gexec, [&] { return run_round(false); }));
    HIPCHK(hipGraphLaunch(gexec, stream));
  }
  const size_t R = (size_t)n_seqs * q.bk;
  HIPCHK(hipMemcpyAsync(h_out, ws + q.out_tok, R * 4, hipMemcpyDeviceToHost, stream));
  HIPCHK(hipMemcpyAsync(h_out + q.R, ws + q.out_n, (size_t)n_seqs * 4, hipMemcpyDeviceToHost, stream));
  HIPCHK(hipMemcpyAsync(h_out + q.R + q.bmax, ws + q.out_a, (size_t)n_seqs * 4, hipMemcpyDeviceToHost, stream));
  HIPCHK(hipStreamSynchronize(stream));
  memcpy(tokens, h_out, R * 4);
  memcpy(n_comm, h_out + q.R, (size_t)n_seqs * 4);
  memcpy(acc, h_out + q.R + q.bmax, (size_t)n_seqs * 4);
  return RT_OK;
}

// The allocation-free round: the kernels of run_round enqueued directly (no graph is
// instantiated), their partial results in the static scratch, the outputs copied to the
// caller's device buffers on the model's stream; no host synchronisation.
int EngineBase::round_static(int32_t* d_tokens, int32_t* d_n_comm, int32_t* d_acc) {
  const Plan& q = p;
  if (q.s_total > kStaticScratchBytes)
    return fail(RT_ERR_CAPACITY, "the configuration's partial results need %zu bytes, beyond the %zu-byte static scratch",
                q.s_total, kStaticScratchBytes);
  if (!prefilled) return fail(RT_ERR_STATE, "rt_spec_round_static called before rt_prefill");
  if (ar_mode) return ar_state_error();
  if (!d_tokens || !d_n_comm || !d_acc) return fail(RT_ERR_INVALID, "null output pointer");
  if (!scratch_dev) return scratch_status != RT_OK ? scratch_status : fail(RT_ERR_HIP, "no static scratch on this device");
  part_base = (char*)scratch_dev;
  // arrival counters start at zero (a kernel, so the call can be captured into a graph)
  fill_zero(part_base + q.s_counters, (size_t)kMaxTiles * 4, stream);
  hipError_t he = hipGetLastError();
  int st = he == hipSuccess ? run_round(false) : fail(RT_ERR_HIP, "fill_zero: %s", hipGetErrorString(he));
  part_base = nullptr;
  if (st != RT_OK) return st;
  const size_t R = (size_t)n_seqs * q.bk;
  HIPCHK(hipMemcpyAsync(d_tokens, ws + q.out_tok, R * 4, hipMemcpyDeviceToDevice, stream));
  HIPCHK(hipMemcpyAsync(d_n_comm, ws + q.out_n, (size_t)n_seqs * 4, hipMemcpyDeviceToDevice, stream));
  HIPCHK(hipMemcpyAsync(d_acc, ws + q.out_a, (size_t)n_seqs * 4, hipMemcpyDeviceToDevice, stream));
  return RT_OK;
}

int EngineBase::profile_round(rt_kernel_stat* stats, double* stage_ms, int32_t* tokens, int32_t* n_comm,
                              int32_t* acc) {
  if (!prefilled) return fail(RT_ERR_STATE, "rt_profile_round called before rt_prefill");
  if (ar_mode) return ar_state_error();
  const Plan& q = p;
  if (ev_pool.empty()) {
    ev_pool.resize(8192);
    for (auto& e : ev_pool) HIPCHK(hipEventCreate(&e));
    for (auto& e : stage_ev) HIPCHK(hipEventCreate(&e));
  }
  std::vector<int32_t> st((size_t)n_seqs * kStateFields);
  HIPCHK(hipStreamSynchronize(stream));
  HIPCHK(hipMemcpy(st.data(), ws + q.state, st.size() * 4, hipMemcpyDeviceToHost));
  prof_ctx.assign(n_seqs, 0);
  for (int s = 0; s < n_seqs; ++s) prof_ctx[s] = st[(size_t)s * kStateFields + ST_SEQ_LEN];
  prof.clear();
  ev_next = 0;
  profiling = true;
  int rc = run_round(false);
  profiling = false;
  launch_events() = LaunchEvents{};
  if (rc != RT_OK) return rc;
  const size_t R = (size_t)n_seqs * q.bk;
  HIPCHK(hipMemcpyAsync(h_out, ws + q.out_tok, R * 4, hipMemcpyDeviceToHost, stream));
  HIPCHK(hipMemcpyAsync(h_out + q.R, ws + q.out_n, (size_t)n_seqs * 4, hipMemcpyDeviceToHost, stream));
  HIPCHK(hipMemcpyAsync(h_out + q.R + q.bmax, ws + q.out_a, (size_t)n_seqs * 4, hipMemcpyDeviceToHost, stream));
  HIPCHK(hipStreamSynchronize(stream));
  memcpy(tokens, h_out, R * 4);
  memcpy(n_comm, h_out + q.R, (size_t)n_seqs * 4);
  memcpy(acc, h_out + q.R + q.bmax, (size_t)n_seqs * 4);
  for (int k = 0; k < RT_K_KINDS; ++k) stats[k] = rt_kernel_stat{k, 0, 0.0, 0.0, 0.0};
  for (const ProfRec& r : prof) {
    float ms = 0.f;
    HIPCHK(hipEventElapsedTime(&ms, r.b, r.e));
    rt_kernel_stat& s = stats[r.kind];
    s.launches += 1;
    s.ms += ms;
    s.bytes += r.bytes;
    s.flops += r.flops;
  }
  for (int i = 0; i < RT_PROF_STAGES; ++i) {
    float ms = 0.f;
    HIPCHK(hipEventElapsedTime(&ms, stage_ev[i], stage_ev[i + 1]));
    stage_ms[i] = ms;
  }
  return RT_OK;
}

// Kernel replay: the launches of one class from a round (with the round's current
// buffers and context lengths) are captured into a graph, replayed `reps` times between
// two HIP events, and averaged.  Only classes whose outputs are per-round scratch are
// allowed, so the replay changes no KV cache and no carried state.
int EngineBase::time_kernel(int kind, int reps, rt_kernel_stat* out) {
  if (!prefilled) return fail(RT_ERR_STATE, "rt_time_kernel called before rt_prefill");
  if (ar_mode) return ar_state_error();
  switch (kind) {
    case RT_K_GEMM_QKV: case RT_K_GEMM_O: case RT_K_GEMM_GATE_UP: case RT_K_GEMM_DOWN:
    case RT_K_GEMM_CONTEXT: case RT_K_GEMM_COND: case RT_K_ATTENTION: case RT_K_ATTN_MERGE:
    case RT_K_LM_HEAD: break;
    default: return fail(RT_ERR_INVALID, "kernel class %d cannot be replayed (it writes KV or round state)", kind);
  }
  if (reps < 1 || reps > 1000) return fail(RT_ERR_INVALID, "reps must be in [1, 1000]");
  const Plan& q = p;
  std::vector<int32_t> st((size_t)n_seqs * kStateFields);
  HIPCHK(hipStreamSynchronize(stream));
  HIPCHK(hipMemcpy(st.data(), ws + q.state, st.size() * 4, hipMemcpyDeviceToHost));
  prof_ctx.assign(n_seqs, 0);
  for (int s = 0; s < n_seqs; ++s) prof_ctx[s] = st[(size_t)s * kStateFields + ST_SEQ_LEN];
  only_kind = kind;
  only_launches = 0;
  only_bytes = only_flops = 0;
  launch_events() = LaunchEvents{};
  launch_events().skip = true;
  hipGraph_t g = nullptr;
  hipError_t be = hipStreamBeginCapture(stream, hipStreamCaptureModeThreadLocal);
  int rc = be == hipSuccess ? run_round(false) : RT_OK;
  hipError_t ce = be == hipSuccess ? hipStreamEndCapture(stream, &g) : be;
  only_kind = -1;
  launch_events() = LaunchEvents{};
  if (rc != RT_OK) { if (g) (void)hipGraphDestroy(g); return rc; }
  if (ce != hipSuccess) { if (g) (void)hipGraphDestroy(g); return fail(RT_ERR_HIP, "replay capture: %s", hipGetErrorString(ce)); }
  hipGraphExec_t ge = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  auto cleanup = [&]() {
    if (ge) (void)hipGraphExecDestroy(ge);
    if (g) (void)hipGraphDestroy(g);
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
  };
  hipError_t e = hipGraphInstantiate(&ge, g, nullptr, nullptr, 0);
  if (e == hipSuccess) e = hipEventCreate(&e0);
  if (e == hipSuccess) e = hipEventCreate(&e1);
  if (e == hipSuccess) e = hipGraphLaunch(ge, stream);          // warm-up
  if (e == hipSuccess) e = hipEventRecord(e0, stream);
  for (int r = 0; r < reps && e == hipSuccess; ++r) e = hipGraphLaunch(ge, stream);
  if (e == hipSuccess) e = hipEventRecord(e1, stream);
  if (e == hipSuccess) e = hipEventSynchronize(e1);
  float ms = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
  cleanup();
  if (e != hipSuccess) return fail(RT_ERR_HIP, "kernel replay: %s", hipGetErrorString(e));
  out->kind = kind;
  out->launches = only_launches;
  out->ms = only_launches ? ms / reps : 0.0;
  out->bytes = only_bytes;
  out->flops = only_flops;
  return RT_OK;
}

static int copy_pages(const EngineBase& m, size_t cache_off, int layer, int seq, bool vlayout, void* dst,
                      size_t bytes, size_t pos0 = 0) {
  const Plan& q = m.p;
  const size_t E = q.esz, hd = q.hd, H = q.Hkv;
  const size_t per_pos = H * hd * E;
  const size_t npos = bytes / per_pos;
  if (bytes % per_pos) return fail(RT_ERR_INVALID, "read of %zu bytes is not a whole number of positions", bytes);
  if (pos0 + npos > (size_t)q.T) return fail(RT_ERR_INVALID, "read past max_seq_len");
  std::vector<int32_t> pt((size_t)q.pages_per_seq);
  HIPCHK(hipMemcpy(pt.data(), m.ws + q.page_table + (size_t)seq * q.pages_per_seq * 4, pt.size() * 4,
                   hipMemcpyDeviceToHost));
  const size_t page_bytes = H * 16 * hd * E;
  std::vector<char> buf(page_bytes);
  char* out = (char*)dst;
  const size_t end = pos0 + npos;
  for (size_t pg = pos0 / 16; pg * 16 < end; ++pg) {
    const char* src = m.ws + cache_off + ((size_t)layer * q.cache_layer_elems) * E + (size_t)pt[pg] * page_bytes;
    HIPCHK(hipMemcpy(buf.data(), src, page_bytes, hipMemcpyDeviceToHost));
    for (size_t t = 0; t < 16; ++t) {
      const size_t pos = pg * 16 + t;
      if (pos < pos0 || pos >= end) continue;
      for (size_t h = 0; h < H; ++h)
        for (size_t e = 0; e < hd; ++e) {
          const size_t si = vlayout ? ((h * hd + e) * 16 + t) : ((h * 16 + t) * hd + e);
          memcpy(out + ((pos - pos0) * H * hd + h * hd + e) * E, buf.data() + si * E, E);
        }
    }
  }
  return RT_OK;
}

// The inverse of copy_pages: positions 0.. of one sequence's cache at `layer`, from
// host rows [pos][Hkv][hd] (each touched page read, patched and written back).
static int write_pages(EngineBase& m, size_t cache_off, int layer, int seq, bool vlayout, const void* src,
                       size_t bytes) {
  const Plan& q = m.p;
  const size_t E = q.esz, hd = q.hd, H = q.Hkv;
  const size_t per_pos = H * hd * E;
  const size_t npos = bytes / per_pos;
  if (bytes % per_pos) return fail(RT_ERR_INVALID, "write of %zu bytes is not a whole number of positions", bytes);
  if (npos > (size_t)q.T) return fail(RT_ERR_INVALID, "write past max_seq_len");
  std::vector<int32_t> pt((size_t)q.pages_per_seq);
  HIPCHK(hipMemcpy(pt.data(), m.ws + q.page_table + (size_t)seq * q.pages_per_seq * 4, pt.size() * 4,
                   hipMemcpyDeviceToHost));
  const size_t page_bytes = H * 16 * hd * E;
  std::vector<char> buf(page_bytes);
  const char* in = (const char*)src;
  for (size_t pg = 0; pg * 16 < npos; ++pg) {
    char* dst = m.ws + cache_off + ((size_t)layer * q.cache_layer_elems) * E + (size_t)pt[pg] * page_bytes;
    HIPCHK(hipMemcpy(buf.data(), dst, page_bytes, hipMemcpyDeviceToHost));
    for (size_t t = 0; t < 16 && pg * 16 + t < npos; ++t)
      for (size_t h = 0; h < H; ++h)
        for (size_t e = 0; e < hd; ++e) {
          const size_t di = vlayout ? ((h * hd + e) * 16 + t) : ((h * 16 + t) * hd + e);
          memcpy(buf.data() + di * E, in + ((pg * 16 + t) * H * hd + h * hd + e) * E, E);
        }
    HIPCHK(hipMemcpy(dst, buf.data(), page_bytes, hipMemcpyHostToDevice));
  }
  return RT_OK;
}

int EngineBase::debug_read(int id, int seq, void* dst, size_t bytes, size_t pos0) {
  const Plan& q = p;
  if (!dst) return fail(RT_ERR_INVALID, "null destination");
  if (seq < 0 || seq >= q.bmax) return fail(RT_ERR_INVALID, "sequence index out of range");
  const bool kv = (id >= RT_T_TARGET_K && id < RT_T_TARGET_K + q.L) || (id >= RT_T_TARGET_V && id < RT_T_TARGET_V + q.L) ||
                  (id >= RT_T_DRAFT_K && id < RT_T_DRAFT_K + q.LD) || (id >= RT_T_DRAFT_V && id < RT_T_DRAFT_V + q.LD);
  if (pos0 && !kv) return fail(RT_ERR_INVALID, "a first position applies to KV cache tensors only");
  size_t off = 0, cap = 0;
  const size_t bk = q.bk;
  if ((id >= RT_T_TRACE_DRAFT_X && id <= RT_T_TRACE_VERIFY_HEAD) || (id >= 1100 && id < 2600))
    return trace_read(id, seq, dst, bytes);
  switch (id) {
    case RT_T_DRAFT_LOGITS: off = q.dlogits + seq * bk * q.V * 4; cap = bk * q.V * 4; break;
    case RT_T_VERIFY_LOGITS: off = q.vlogits + seq * bk * q.V * 4; cap = bk * q.V * 4; break;
    case RT_T_HD: off = q.hd_keep + seq * bk * q.d * q.ksz; cap = bk * q.d * q.ksz; break;
    case RT_T_HT: off = q.ht_keep + seq * bk * q.d * q.ksz; cap = bk * q.d * q.ksz; break;
    case RT_T_ETILDE: off = q.etilde + seq * bk * q.d * 4; cap = bk * q.d * 4; break;
    case RT_T_DRAFT_TOKENS: off = q.dtok + seq * bk * 4; cap = bk * 4; break;
    case RT_T_TARGET_TOKENS: off = q.ttok + seq * bk * 4; cap = bk * 4; break;
    case RT_T_STATE: off = q.state + (size_t)seq * kStateFields * 4; cap = kStateFields * 4; break;
    case RT_T_AR_LOGITS: off = q.vlogits + seq * (size_t)q.V * 4; cap = (size_t)q.V * 4; break;
    case RT_T_DRAFT_DIST_IDS: off = q.dist_ids_d + seq * bk * RT_MAX_TOP_K * 4; cap = bk * RT_MAX_TOP_K * 4; break;
    case RT_T_DRAFT_DIST_P: off = q.dist_p_d + seq * bk * RT_MAX_TOP_K * 4; cap = bk * RT_MAX_TOP_K * 4; break;
    case RT_T_VERIFY_DIST_IDS: off = q.dist_ids_v + seq * bk * RT_MAX_TOP_K * 4; cap = bk * RT_MAX_TOP_K * 4; break;
    case RT_T_VERIFY_DIST_P: off = q.dist_p_v + seq * bk * RT_MAX_TOP_K * 4; cap = bk * RT_MAX_TOP_K * 4; break;
    case RT_T_G: {
      // packed [group][k tile][lane][8] -> row-major [bk][n_cond * d]
      const size_t ncd = (size_t)q.nc * q.d, ldg = (size_t)16 * q.Kp_nc;
      if (bytes > bk * ncd * q.esz) return fail(RT_ERR_INVALID, "read too large");
      const int r0 = seq * q.bk, r1 = r0 + q.bk;
      const int g0 = r0 / 16, g1 = (r1 + 15) / 16;
      std::vector<char> buf((size_t)(g1 - g0) * ldg * q.esz);
      HIPCHK(hipStreamSynchronize(stream));
      HIPCHK(hipMemcpy(buf.data(), ws + q.g + (size_t)g0 * ldg * q.esz, buf.size(), hipMemcpyDeviceToHost));
      char* out = (char*)dst;
      const size_t nrow = bytes / (ncd * q.esz);
      for (size_t r = 0; r < nrow; ++r)
        for (size_t k = 0; k < ncd; ++k)
          memcpy(out + (r * ncd + k) * q.esz, buf.data() + (pa_index((int)(r0 + r), (int)k, ldg) - (size_t)g0 * ldg) * q.esz,
                 q.esz);
      return RT_OK;
    }
    default: {
      HIPCHK(hipStreamSynchronize(stream));
      if (id >= RT_T_TARGET_K && id < RT_T_TARGET_K + q.L) return copy_pages(*this, q.kc, id - RT_T_TARGET_K, seq, false, dst, bytes, pos0);
      if (id >= RT_T_TARGET_V && id < RT_T_TARGET_V + q.L) return copy_pages(*this, q.vc, id - RT_T_TARGET_V, seq, true, dst, bytes, pos0);
      if (id >= RT_T_DRAFT_K && id < RT_T_DRAFT_K + q.LD) return copy_pages(*this, q.dkc, id - RT_T_DRAFT_K, seq, false, dst, bytes, pos0);
      if (id >= RT_T_DRAFT_V && id < RT_T_DRAFT_V + q.LD) return copy_pages(*this, q.dvc, id - RT_T_DRAFT_V, seq, true, dst, bytes, pos0);
      return fail(RT_ERR_INVALID, "unknown tensor id %d", id);
    }
  }
  if (bytes > cap) return fail(RT_ERR_INVALID, "read of %zu bytes exceeds %zu", bytes, cap);
  HIPCHK(hipStreamSynchronize(stream));
  HIPCHK(hipMemcpy(dst, ws + off, bytes, hipMemcpyDeviceToHost));
  return RT_OK;
}

int EngineBase::trace_read(int id, int seq, void* dst, size_t bytes) {
  const Plan& q = p;
  if (!trace) return fail(RT_ERR_STATE, "the layer trace is off (debug flag 8)");
  int rec = -1, it = TI_X;
  if (id >= RT_T_TRACE_DRAFT_X && id <= RT_T_TRACE_DRAFT_X + q.LD) {
    const int l = id - RT_T_TRACE_DRAFT_X;
    rec = l < q.LD ? l : q.LD + q.L;
  } else if (id >= RT_T_TRACE_TARGET_X && id <= RT_T_TRACE_TARGET_X + q.L) {
    const int l = id - RT_T_TRACE_TARGET_X;
    rec = l < q.L ? q.LD + l : q.LD + q.L + 1;
  } else if (id == RT_T_TRACE_DRAFT_HEAD || id == RT_T_TRACE_VERIFY_HEAD) {
    rec = q.LD + q.L + (id == RT_T_TRACE_VERIFY_HEAD);
    it = TI_H2;
  } else if (id >= 1100 && id < 2600) {
    const int pass = id / 1000, kind = (id % 1000) / 100, l = id % 100;
    if (kind >= 1 && kind < TI_COUNT && l < (pass == 1 ? q.LD : q.L)) {
      rec = pass == 1 ? l : q.LD + l;
      it = kind;
    }
  }
  if (rec < 0) return fail(RT_ERR_INVALID, "unknown tensor id %d", id);
  const size_t bk = q.bk, E = q.esz;
  const size_t width = it == TI_Q || it == TI_ATTN ? (size_t)q.qN : it == TI_MLP ? (size_t)q.F : (size_t)q.d;
  const size_t esz = it == TI_X || it == TI_XMID ? 4 : E;
  if (bytes > bk * width * esz) return fail(RT_ERR_INVALID, "read of %zu bytes exceeds %zu", bytes, bk * width * esz);
  HIPCHK(hipStreamSynchronize(stream));
  const char* base = trace + (size_t)rec * trace_rec_bytes + trace_item_off[it];
  if (it == TI_X || it == TI_XMID || it == TI_Q) {   // row-major [R][width]
    HIPCHK(hipMemcpy(dst, base + (size_t)seq * bk * width * esz, bytes, hipMemcpyDeviceToHost));
    return RT_OK;
  }
  // packed GEMM operand (16-row groups) -> row-major [bk][width]
  const int Kp = it == TI_ATTN ? q.Kp_q : it == TI_MLP ? q.Kp_F : q.Kp_d;
  const size_t ldg = (size_t)16 * Kp;
  std::vector<char> buf(trace_item_bytes(it));
  HIPCHK(hipMemcpy(buf.data(), base, buf.size(), hipMemcpyDeviceToHost));
  char* out = (char*)dst;
  const size_t nrow = bytes / (width * E);
  for (size_t r = 0; r < nrow; ++r)
    for (size_t k = 0; k < width; ++k)
      memcpy(out + (r * width + k) * E, buf.data() + pa_index((int)(seq * bk + r), (int)k, ldg) * E, E);
  return RT_OK;
}

int EngineBase::debug_write(int id, int seq, const void* src, size_t bytes) {
  const Plan& q = p;
  if (!src) return fail(RT_ERR_INVALID, "null source");
  if (seq < 0 || seq >= q.bmax) return fail(RT_ERR_INVALID, "sequence index out of range");
  size_t off = 0, cap = 0;
  const size_t bk = q.bk;
  switch (id) {
    case RT_T_HD: off = q.hd_keep + seq * bk * q.d * q.ksz; cap = bk * q.d * q.ksz; break;
    case RT_T_HT: off = q.ht_keep + seq * bk * q.d * q.ksz; cap = bk * q.d * q.ksz; break;
    case RT_T_STATE: off = q.state + (size_t)seq * kStateFields * 4; cap = kStateFields * 4; break;
    default: {
      HIPCHK(hipStreamSynchronize(stream));
      if (id >= RT_T_TARGET_K && id < RT_T_TARGET_K + q.L) return write_pages(*this, q.kc, id - RT_T_TARGET_K, seq, false, src, bytes);
      if (id >= RT_T_TARGET_V && id < RT_T_TARGET_V + q.L) return write_pages(*this, q.vc, id - RT_T_TARGET_V, seq, true, src, bytes);
      if (id >= RT_T_DRAFT_K && id < RT_T_DRAFT_K + q.LD) return write_pages(*this, q.dkc, id - RT_T_DRAFT_K, seq, false, src, bytes);
      if (id >= RT_T_DRAFT_V && id < RT_T_DRAFT_V + q.LD) return write_pages(*this, q.dvc, id - RT_T_DRAFT_V, seq, true, src, bytes);
      return fail(RT_ERR_INVALID, "tensor id %d is not writable", id);
    }
  }
  if (bytes > cap) return fail(RT_ERR_INVALID, "write of %zu bytes exceeds %zu", bytes, cap);
  HIPCHK(hipStreamSynchronize(stream));
  HIPCHK(hipMemcpy(ws + off, src, bytes, hipMemcpyHostToDevice));
  return RT_OK;
}

}  // namespace rt

struct rt_model {
  rt::EngineBase* e;
};

using namespace rt;

extern "C" {

size_t rt_workspace_bytes(const rt_config* cfg) {
  Plan p;
  if (make_plan(cfg, &p) != RT_OK) return 0;
  return p.total;
}

int32_t rt_weight_count(const rt_config* cfg) {
  if (validate_config(cfg) != RT_OK) return 0;
  return weight_count(cfg);
}

int64_t rt_weight_elements(const rt_config* cfg, int32_t index) {
  if (validate_config(cfg) != RT_OK) return 0;
  return (int64_t)weight_elems(cfg, index);
}

int rt_init_models(const rt_config* cfg, const void* const* weights, int32_t n_weights, void* d_workspace,
                   size_t ws_bytes, void* hip_stream, rt_model** out) {
  try {
    if (!out) return fail(RT_ERR_INVALID, "out handle pointer is null");
    *out = nullptr;
    Plan p;
    int st = make_plan(cfg, &p);
    if (st) return st;
    if (!weights) return fail(RT_ERR_INVALID, "weights is null");
    if (n_weights != weight_count(cfg))
      return fail(RT_ERR_INVALID, "expected %d weight tensors, got %d", weight_count(cfg), n_weights);
    for (int i = 0; i < n_weights; ++i)
      if (!weights[i]) return fail(RT_ERR_INVALID, "weight %d is null", i);
    if (!d_workspace) return fail(RT_ERR_WORKSPACE, "workspace is null");
    if ((uintptr_t)d_workspace % 256) return fail(RT_ERR_WORKSPACE, "workspace must be 256-byte aligned");
    if (ws_bytes < p.total) return fail(RT_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, p.total);
    EngineBase* e = nullptr;
    if (cfg->dtype == RT_BF16) e = new (std::nothrow) Engine<bf16_t, uint16_t>();
    else e = new (std::nothrow) Engine<float, float>();
    if (!e) return fail(RT_ERR_INVALID, "out of host memory");
    e->cfg = *cfg;
    e->p = p;
    e->ws = (char*)d_workspace;
    {
      hipError_t de = hipGetDevice(&e->device);
      if (de != hipSuccess) { delete e; return fail(RT_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(de)); }
      // the static scratch's device address, looked up once per device with it current
      e->scratch_status = scratch_setup(e->device, &e->scratch_dev);
      if (e->scratch_status != RT_OK) e->scratch_dev = nullptr;
    }
    if (hip_stream) {
      e->stream = (hipStream_t)hip_stream;
    } else {
      hipError_t he = hipStreamCreateWithFlags(&e->stream, hipStreamNonBlocking);
      if (he != hipSuccess) { delete e; return fail(RT_ERR_HIP, "hipStreamCreate: %s", hipGetErrorString(he)); }
      e->own_stream = true;
    }
    hipError_t he = hipHostMalloc((void**)&e->h_out, ((size_t)p.R + 3 * (size_t)p.bmax) * 4, hipHostMallocDefault);
    if (he != hipSuccess) { delete e; return fail(RT_ERR_HIP, "hipHostMalloc: %s", hipGetErrorString(he)); }
    // weights in host memory (pageable or pinned) go through temporary device copies,
    // released once the packing on the stream has finished
    struct Staged {
      std::vector<void*> b;
      hipStream_t s = nullptr;
      ~Staged() {
        if (s) (void)hipStreamSynchronize(s);
        for (void* x : b) (void)hipFree(x);
      }
    } staged;
    staged.s = e->stream;
    std::vector<const void*> wdev(weights, weights + n_weights);
    for (int i = 0; i < n_weights; ++i) {
      hipPointerAttribute_t at{};
      const hipError_t pe = hipPointerGetAttributes(&at, weights[i]);
      if (pe != hipSuccess) (void)hipGetLastError();   // unregistered host memory
      if (pe == hipSuccess && (at.type == hipMemoryTypeDevice || at.type == hipMemoryTypeManaged)) continue;
      const size_t bytes = weight_elems(cfg, i) * (cfg->dtype == RT_BF16 ? 2 : 4);
      void* b = nullptr;
      hipError_t ae = hipMalloc(&b, bytes);
      if (ae == hipSuccess) {
        staged.b.push_back(b);
        ae = hipMemcpy(b, weights[i], bytes, hipMemcpyHostToDevice);
      }
      if (ae != hipSuccess) {
        staged.s = nullptr;   // nothing was enqueued yet
        delete e;
        return fail(RT_ERR_HIP, "uploading host weight %d: %s", i, hipGetErrorString(ae));
      }
      wdev[i] = b;
    }
    st = e->init(wdev.data());
    if (st) {
      (void)hipStreamSynchronize(e->stream);   // packing kernels done before the copies go
      staged.s = nullptr;
      delete e;
      return st;
    }
    rt_model* m = new (std::nothrow) rt_model{e};
    if (!m) { delete e; return fail(RT_ERR_INVALID, "out of host memory"); }
    *out = m;
    return RT_OK;
  } catch (...) {
    return fail(RT_ERR_INVALID, "unexpected exception in rt_init_models");
  }
}

int rt_prefill(rt_model* m, int32_t n_seqs, const int32_t* prompt_lens, const int32_t* prompt_ids,
               int32_t gen_budget, int32_t* first_tokens) {
  try {
    if (!m || !m->e) return fail(RT_ERR_INVALID, "null model");
    EngineBase& e = *m->e;
    if (!prompt_lens || !prompt_ids || !first_tokens) return fail(RT_ERR_INVALID, "null pointer argument");
    if (n_seqs < 1 || n_seqs > e.p.bmax) return fail(RT_ERR_CAPACITY, "n_seqs %d outside [1, %d]", n_seqs, e.p.bmax);
    if (gen_budget < 1) return fail(RT_ERR_INVALID, "gen_budget must be >= 1");
    size_t total = 0;
    for (int s = 0; s < n_seqs; ++s) {
      const int len = prompt_lens[s];
      if (len < 1) return fail(RT_ERR_INVALID, "prompt %d is empty", s);
      if ((long long)len + gen_budget + e.p.bk > e.p.T)
        return fail(RT_ERR_CAPACITY, "prompt %d: length %d + budget %d + block %d exceeds max_seq_len %d", s, len,
                    gen_budget, e.p.bk, e.p.T);
      total += (size_t)len;
    }
    for (size_t i = 0; i < total; ++i)
      if (prompt_ids[i] < 0 || prompt_ids[i] >= e.p.V) return fail(RT_ERR_TOKEN, "prompt token %d out of range", prompt_ids[i]);
    return e.prefill(n_seqs, prompt_lens, prompt_ids, gen_budget, first_tokens);
  } catch (...) {
    return fail(RT_ERR_INVALID, "unexpected exception in rt_prefill");
  }
}

int rt_spec_round(rt_model* m, int32_t* tokens, int32_t* n_committed, int32_t* accept_len) {
  try {
    if (!m || !m->e) return fail(RT_ERR_INVALID, "null model");
    return m->e->round(nullptr, tokens, n_committed, accept_len);
  } catch (...) {
    return fail(RT_ERR_INVALID, "unexpected exception in rt_spec_round");
  }
}

int rt_spec_round_forced(rt_model* m, const int32_t* drafts, int32_t* tokens, int32_t* n_committed,
                         int32_t* accept_len) {
  try {
    if (!m || !m->e) return fail(RT_ERR_INVALID, "null model");
    if (!drafts) return fail(RT_ERR_INVALID, "null drafts");
    return m->e->round(drafts, tokens, n_committed, accept_len);
  } catch (...) {
    return fail(RT_ERR_INVALID, "unexpected exception in rt_spec_round_forced");
  }
}

int rt_spec_round_static(rt_model* m, int32_t* d_tokens, int32_t* d_n_committed, int32_t* d_accept_len) {
  try {
    if (!m || !m->e) return fail(RT_ERR_INVALID, "null model");
    return m->e->round_static(d_tokens, d_n_committed, d_accept_len);
  } catch (...) {
    return fail(RT_ERR_INVALID, "unexpected exception in rt_spec_round_static");
  }
}

int rt_profile_round(rt_model* m, rt_kernel_stat* stats, double* stage_ms, int32_t* tokens,
                     int32_t* n_committed, int32_t* accept_len) {
  try {
    if (!m || !m->e) return fail(RT_ERR_INVALID, "null model");
    if (!stats || !stage_ms || !tokens || !n_committed || !accept_len) return fail(RT_ERR_INVALID, "null pointer argument");
    return m->e->profile_round(stats, stage_ms, tokens, n_committed, accept_len);
  } catch (...) {
    return fail(RT_ERR_INVALID, "unexpected exception in rt_profile_round");
  }
}

int rt_ar_steps(rt_model* m, int32_t n_steps, int32_t* tokens, int32_t* n_generated) {
  try {
    if (!m || !m->e) return fail(RT_ERR_INVALID, "null model");
    return m->e->ar_steps(n_steps, tokens, n_generated);
  } catch (...) {
    return fail(RT_ERR_INVALID, "unexpected exception in rt_ar_steps");
  }
}

int rt_time_kernel(rt_model* m, int32_t kind, int32_t reps, rt_kernel_stat* stat) {
  try {
    if (!m || !m->e) return fail(RT_ERR_INVALID, "null model");
    if (!stat) return fail(RT_ERR_INVALID, "null pointer argument");
    return m->e->time_kernel(kind, reps, stat);
  } catch (...) {
    return fail(RT_ERR_INVALID, "unexpected exception in rt_time_kernel");
  }
}

int rt_stream_read(const void* d_buf, size_t buf_bytes, size_t bytes, int32_t grid, int32_t reps, void* hip_stream,
                   double* us) {
  try {
    if (!d_buf || !us) return fail(RT_ERR_INVALID, "null pointer argument");
    if (bytes < 16 || bytes % 16 || (uintptr_t)d_buf % 256)
      return fail(RT_ERR_INVALID, "bytes must be a positive multiple of 16 and the buffer 256-byte aligned");
    if (bytes > buf_bytes) return fail(RT_ERR_INVALID, "bytes exceed the buffer");
    if (grid < 1 || grid > 65536) return fail(RT_ERR_INVALID, "grid must be in [1, 65536]");
    if (reps < 1 || reps > 1000) return fail(RT_ERR_INVALID, "reps must be in [1, 1000]");
    hipStream_t s = (hipStream_t)hip_stream;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    uint32_t* sink = nullptr;
    hipError_t e = hipEventCreate(&e0);
    if (e == hipSuccess) e = hipEventCreate(&e1);
    // the sink is never written (its store is switched off at launch); the buffer serves
    if (e == hipSuccess) sink = (uint32_t*)d_buf;
    // launch r reads the window at ((r + 1) * bytes) mod (buf_bytes - bytes + 1), 256-byte
    // aligned, so consecutive launches read different data (a window read again comes
    // buf_bytes / bytes launches later, after the 256 MB memory-side cache has turned over)
    const size_t span = buf_bytes - bytes + 1;
    auto window = [&](int r) { return (const char*)d_buf + ((((size_t)r + 1) * bytes) % span & ~(size_t)255); };
    if (e == hipSuccess) { stream_read(d_buf, bytes, grid, sink, s); e = hipGetLastError(); }   // warm-up
    if (e == hipSuccess) e = hipEventRecord(e0, s);
    for (int r = 0; r < reps && e == hipSuccess; ++r) { stream_read(window(r), bytes, grid, sink, s); e = hipGetLastError(); }
    if (e == hipSuccess) e = hipEventRecord(e1, s);
    if (e == hipSuccess) e = hipEventSynchronize(e1);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
    if (e != hipSuccess) return fail(RT_ERR_HIP, "stream read: %s", hipGetErrorString(e));
    *us = (double)ms * 1e3 / reps;
    return RT_OK;
  } catch (...) {
    return fail(RT_ERR_INVALID, "unexpected exception in rt_stream_read");
  }
}

int rt_set_debug(rt_model* m, int32_t flags) {
  if (!m || !m->e) return fail(RT_ERR_INVALID, "null model");
  if (flags < 0 || flags > 127) return fail(RT_ERR_INVALID, "unknown debug flags %d", flags);
  if (flags & 8) {
    const int st = m->e->alloc_trace();
    if (st) return st;
  }
  m->e->flags = flags;
  m->e->drop_graph();
  return RT_OK;
}

int rt_debug_read(rt_model* m, int32_t tensor_id, int32_t seq, void* host_dst, size_t bytes) {
  try {
    if (!m || !m->e) return fail(RT_ERR_INVALID, "null model");
    return m->e->debug_read(tensor_id, seq, host_dst, bytes);
  } catch (...) {
    return fail(RT_ERR_INVALID, "unexpected exception in rt_debug_read");
  }
}

int rt_debug_read_rows(rt_model* m, int32_t tensor_id, int32_t seq, int32_t pos0, void* host_dst, size_t bytes) {
  try {
    if (!m || !m->e) return fail(RT_ERR_INVALID, "null model");
    if (pos0 < 0) return fail(RT_ERR_INVALID, "negative first position");
    return m->e->debug_read(tensor_id, seq, host_dst, bytes, (size_t)pos0);
  } catch (...) {
    return fail(RT_ERR_INVALID, "unexpected exception in rt_debug_read_rows");
  }
}

int rt_debug_write(rt_model* m, int32_t tensor_id, int32_t seq, const void* host_src, size_t bytes) {
  try {
    if (!m || !m->e) return fail(RT_ERR_INVALID, "null model");
    return m->e->debug_write(tensor_id, seq, host_src, bytes);
  } catch (...) {
    return fail(RT_ERR_INVALID, "unexpected exception in rt_debug_write");
  }
}

int rt_destroy(rt_model* m) {
  if (!m) return fail(RT_ERR_INVALID, "null model");
  if (m->e) (void)hipStreamSynchronize(m->e->stream);
  delete m->e;
  delete m;
  return RT_OK;
}

const char* rt_last_error(void) { return rt::last_error(); }

}  // extern "C"
