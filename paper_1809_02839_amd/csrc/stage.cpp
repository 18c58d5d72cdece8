// Stage engine: owns the float32 W / v / g arenas, the two predicted-weight
// slots, the activation stash ring (one slot per mini-batch in flight) and a
// workspace, and turns forward / backward / update calls into kernel launches
// on the stage's stream. The per-kind sequences follow the layer definitions
// of the five workload kinds (Section 4.1 of the paper: VGG-style 3x3
// convolutions, ResNet bottlenecks, a post-LN Transformer encoder, a residual
// LSTM, and fully-connected layers), with the forward pass reading predicted
// slot 0 and the backward pass reading slot 1 (Section 3.2, Eq. 5 and Eq. 6).
#include "stage.hpp"

#include <algorithm>
#include <cmath>
#include <cstring>

namespace spx {

void hip_check(hipError_t e, const char* what) {
  if (e != hipSuccess) throw StageError(SPECTRAIN_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

// ------------------------------------------------------------ DeviceBlock ----
size_t DeviceBlock::add(size_t bytes) {
  size_t off = total_;
  total_ += (bytes + 255) & ~static_cast<size_t>(255);
  return off;
}
void DeviceBlock::allocate() {
  if (total_ == 0) return;
  void* p = nullptr;
  hipError_t e = hipMalloc(&p, total_);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    throw StageError(SPECTRAIN_ENOMEM, "hipMalloc of " + std::to_string(total_) + " bytes failed: " +
                                           hipGetErrorString(e));
  }
  base_ = static_cast<char*>(p);
}
void DeviceBlock::release() {
  if (base_) (void)hipFree(base_);
  base_ = nullptr;
}

void PinnedInts::allocate(size_t n) {
  hip_check(hipHostMalloc(reinterpret_cast<void**>(&host_), n * sizeof(int), hipHostMallocMapped), "hipHostMalloc");
  for (size_t i = 0; i < n; ++i) host_[i] = 0;
  hip_check(hipHostGetDevicePointer(reinterpret_cast<void**>(&dev_), host_, 0), "hipHostGetDevicePointer");
}

PinnedInts::~PinnedInts() {
  if (host_) (void)hipHostFree(host_);
}

namespace {

constexpr long TENSOR_ALIGN = 64;   // elements: 256 B of float32, 128 B of bf16
constexpr float LN_EPS = 1e-5f;

Operand opK(const void* p, long ld) {
  Operand o;
  o.ptr = p;
  o.ld = ld;
  o.mode = OP_K_PLAIN;
  return o;
}
Operand opR(const void* p, long ld) {
  Operand o;
  o.ptr = p;
  o.ld = ld;
  o.mode = OP_R_PLAIN;
  return o;
}
Operand opConv(int mode, const void* p, int B, int H, int W, int C, int C2 = 0) {
  Operand o;
  o.ptr = p;
  o.mode = mode;
  o.g.B = B;
  o.g.H = H;
  o.g.W = W;
  o.g.C = C;
  o.g.C2 = C2;
  return o;
}
GemmDesc gd(int M, int N, int K, const Operand& A, const Operand& B, long ldc) {
  GemmDesc d;
  d.M = M;
  d.N = N;
  d.K = K;
  d.A = A;
  d.B = B;
  d.epi.ldc = ldc;
  return d;
}

void fail(const std::string& m) { throw StageError(SPECTRAIN_EINVAL, m); }

// Algorithmic bytes of the elementwise and row passes (one read of each
// input, one write of each output).
double ce_bytes(double R, double C) { return R * C * (4.0 + 2.0) + R * 8.0; }   // scores, gradient, label, loss
double colsum_bytes(double R, double C, double esz) { return R * C * esz + C * 4.0; }
double ln_bytes(double R, double D) { return R * D * 4.0 + R * 8.0 + D * 4.0; }  // r in, y out (bf16), stats
double lnb_rows_bytes(double R, double D) { return R * D * 6.0 + R * 8.0 + D * 2.0; }   // dy, r in, dr out, stats
double lnb_params_bytes(double R, double D) {   // per-block partials of 3 column sums in, 3 sums out
  return 12.0 * D * ((R + LNB_ROWS - 1) / LNB_ROWS) + 12.0 * D;
}

}  // namespace

// ----------------------------------------------------------------- layout ----
void Stage::build_layout() {
  const int* dm = d_.dims;
  const int L = d_.num_layers;
  std::vector<long> sizes;
  switch (d_.kind) {
    case SPECTRAIN_KIND_FC: {
      for (int l = 0; l < L; ++l) {
        long fin = l == 0 ? dm[0] : dm[2];
        long fout = l == L - 1 ? dm[1] : dm[2];
        sizes.push_back(fout * fin);
        sizes.push_back(fout);
      }
      break;
    }
    case SPECTRAIN_KIND_CONV3X3:
      for (int l = 0; l < L; ++l) sizes.push_back(static_cast<long>(dm[1]) * 9 * (l == 0 ? dm[0] : dm[1]));
      if (d_.head == SPECTRAIN_HEAD_CE) {   // classifier [classes, C_out] and its bias
        sizes.push_back(static_cast<long>(dm[4]) * dm[1]);
        sizes.push_back(dm[4]);
      }
      break;
    case SPECTRAIN_KIND_BOTTLENECK:
      for (int l = 0; l < L; ++l) {
        sizes.push_back(static_cast<long>(dm[1]) * dm[0]);
        sizes.push_back(static_cast<long>(dm[1]) * 9 * dm[1]);
        sizes.push_back(static_cast<long>(dm[0]) * dm[1]);
      }
      if (d_.head == SPECTRAIN_HEAD_CE) {   // classifier [classes, C] and its bias
        sizes.push_back(static_cast<long>(dm[4]) * dm[0]);
        sizes.push_back(dm[4]);
      }
      break;
    case SPECTRAIN_KIND_TRANSFORMER: {
      const long d = dm[0], F = dm[2];
      for (int l = 0; l < L; ++l) {
        long s[12] = {3 * d * d, 3 * d, d * d, d, d, d, F * d, F, d * F, d, d, d};
        sizes.insert(sizes.end(), s, s + 12);
      }
      if (d_.head == SPECTRAIN_HEAD_CE) {   // vocabulary projection [V, d] and its bias
        sizes.push_back(static_cast<long>(dm[4]) * d);
        sizes.push_back(dm[4]);
      }
      break;
    }
    case SPECTRAIN_KIND_RESLSTM: {
      const long I = dm[0], H = dm[1], V = dm[3];
      for (int l = 0; l < L; ++l) {
        sizes.push_back(4 * H * (l == 0 ? I : H));
        sizes.push_back(4 * H * H);
        sizes.push_back(4 * H);
      }
      if (d_.head == SPECTRAIN_HEAD_CE) {
        sizes.push_back(V * H);
        sizes.push_back(V);
      }
      break;
    }
    default:
      fail("unknown stage kind");
  }
  long off = 0;
  n_params_ = 0;
  for (long n : sizes) {
    tensors_.push_back({off, n});
    off += (n + TENSOR_ALIGN - 1) / TENSOR_ALIGN * TENSOR_ALIGN;
    n_params_ += n;
  }
  n_arena_ = off;
}

const void* Stage::wf(int i) const { return static_cast<const char*>(what_[0]) + tensors_[i].off * esz_; }
const void* Stage::wb(int i) const { return static_cast<const char*>(bwd_weights_) + tensors_[i].off * esz_; }

// Algorithmic HBM bytes of one GEMM launch: each operand tensor read once
// (a convolution gather reads its feature map once, not once per tap), the
// outputs written once (read too when accumulating), and every epilogue
// operand (bias, residual, mask) read once. Split-K partials are not counted:
// they are traffic of the implementation, not of the product.
double gemm_algorithmic_bytes(const GemmDesc& d, size_t esz) {
  auto operand = [&](const Operand& o, long rows) -> double {
    switch (o.mode) {
      case OP_K_PLAIN:
      case OP_R_PLAIN: return static_cast<double>(rows) * d.K * esz;
      case OP_R_FILTER_T: return 9.0 * o.g.C * o.g.C2 * esz;
      default: return static_cast<double>(o.g.B) * o.g.H * o.g.W * o.g.C * esz;
    }
  };
  const Epilogue& e = d.epi;
  double per_out = 0.0;
  if (e.out_f32) per_out += e.accumulate ? 8.0 : 4.0;
  if (e.out_bf16) per_out += 2.0;
  if (e.res_f32) per_out += 4.0;
  if (e.res_bf16) per_out += 2.0;
  if (e.mask) per_out += static_cast<double>(esz);
  double b = operand(d.A, d.M) + operand(d.B, d.N) + static_cast<double>(d.M) * d.N * per_out;
  if (e.bias) b += 4.0 * d.N;
  else if (e.bias_bf16) b += 2.0 * d.N;
  return b * d.batch;
}

void Stage::gemm(const GemmDesc& d, bool defer) {
  // launch families are the kernel instantiations, as a profiler names them
  // (names and work are only worked out while profiling: they cost host time)
  const double flops = 2.0 * d.M * d.N * static_cast<double>(d.K) * d.batch;
  const double bytes = prof_on_ ? gemm_algorithmic_bytes(d, esz_) : 0.0;
  GemmDesc dd = d;
  const bool side = ls_ == s2_;   // each stream has its own split-K partials
  dd.workspace = ext_ws_ ? ext_ws_ + (side ? gemm_ws_bytes_ / 4 : 0) : ws<float>(side ? ws_split2_ : ws_split_);
  dd.workspace_bytes = gemm_ws_bytes_;
  dd.concurrent = concurrent_;
  if (!dt_) {
    LAUNCH(prof_on_ ? gemm_f32_kernel_name(dd) : "gemm_f32", flops, bytes, gemm_f32(dd, ls_));
    return;
  }
  if (defer) {
    const Epilogue& e = d.epi;
    const long mn = static_cast<long>(d.M) * d.N;
    const long off = e.out_f32 ? static_cast<long>(e.out_f32 - g_) : -1;
    const bool plain = d.batch == 1 && e.out_f32 && !e.out_bf16 && !e.bias && !e.bias_bf16 && !e.res_f32 &&
                       !e.res_bf16 && !e.mask && e.alpha == 1.0f && !e.relu && !e.accumulate && e.ldc == d.N;
    const int splits = gemm_bf16_split_rule(d.M, d.N, d.K, d.batch, gemm_ws_bytes_, concurrent_);
    if (plain && splits > 1 && off >= 0 && off + mn <= n_arena_ && off % 8 == 0 && mn % 8 == 0 &&
        defer_used_ + splits * mn <= defer_cap_ && defer_segs_.size() < static_cast<size_t>(UPDATE_MAX_SEGMENTS)) {
      dd.workspace = defer_ + defer_used_;
      dd.workspace_bytes = static_cast<size_t>(splits * mn) * 4;
      // the partial planes replace the g write: splits - 1 planes more
      LAUNCH_X(prof_on_ ? gemm_bf16_kernel_name(dd) : "gemm_bf16", flops, bytes, 4.0 * (splits - 1) * mn,
               gemm_bf16(dd, ls_, GEMM_MAIN));
      UpdateSegment sg;
      sg.off = off;
      sg.n = mn;
      sg.part = dd.workspace;
      sg.splits = splits;
      defer_segs_.push_back(sg);
      defer_used_ += splits * mn;
      return;
    }
  }
  const int splits = gemm_bf16_splits(dd);
  const double mn = static_cast<double>(d.M) * d.N * d.batch;
  // with a K split the GEMM writes float32 partial planes instead of the output
  LAUNCH_X(prof_on_ ? gemm_bf16_kernel_name(dd) : "gemm_bf16", flops, bytes, splits > 1 ? 4.0 * splits * mn : 0.0,
           gemm_bf16(dd, ls_, GEMM_MAIN));
  if (splits > 1) {
    // the reduction's own traffic: partials read once, output written once
    // (read too when accumulating), epilogue operands read once
    const double out = d.epi.out_f32 ? 4.0 : 2.0;
    const double rbytes = mn * (4.0 * splits + out * (d.epi.accumulate ? 2 : 1));
    LAUNCH(prof_on_ ? gemm_bf16_reduce_name(dd) : "splitk_reduce", 0, rbytes, gemm_bf16(dd, ls_, GEMM_REDUCE));
  }
}

void Stage::side_gemm(const GemmDesc& d, std::initializer_list<const void*> reads) {
  on_side(reads, [&]() { gemm(d); });
}

void Stage::protect(const void* buf) {
  auto it = side_reads_.find(buf);
  if (it == side_reads_.end()) return;
  hip_check(hipStreamWaitEvent(s_, it->second, 0), "hipStreamWaitEvent");
  side_reads_.erase(it);
}

void Stage::join_side() {
  side_reads_.clear();
  if (!side_pending_) return;
  hip_check(hipEventRecord(join_ev_, s2_), "hipEventRecord");
  hip_check(hipStreamWaitEvent(s_, join_ev_, 0), "hipStreamWaitEvent");
  side_pending_ = false;
}

// ------------------------------------------------------------ profiling ----
hipEvent_t Stage::prof_event() {
  if (prof_used_ == prof_pool_.size()) {
    hipEvent_t e;
    hip_check(hipEventCreate(&e), "hipEventCreate");
    prof_pool_.push_back(e);
  }
  return prof_pool_[prof_used_++];
}

void Stage::prof_collect() {
  if (prof_recs_.empty()) return;
  sync();
  for (const ProfRec& r : prof_recs_) {
    float ms = 0.0f;
    hip_check(hipEventElapsedTime(&ms, r.a, r.b), "hipEventElapsedTime");
    spectrain_kernel_stat& k = prof_stats_[r.family];
    k.launches += 1;
    k.ms_total += ms;
    k.flops_total += r.flops;
    k.bytes_total += r.bytes;
    k.extra_bytes_total += r.extra;
  }
  prof_recs_.clear();
  prof_used_ = 0;
}

void Stage::profile(bool enable, bool serial) {
  if (enable) {
    prof_collect();
    prof_stats_.clear();
    prof_index_.clear();
  }
  prof_on_ = enable;
  serial_ = enable && serial;
}

int Stage::profile_read(spectrain_kernel_stat* out, int capacity) {
  prof_collect();
  const int n = static_cast<int>(prof_stats_.size());
  for (int i = 0; i < n && i < capacity; ++i) out[i] = prof_stats_[i];
  return n;
}


// Sizes of the stash slot buffers and workspace buffers of each kind.
void Stage::plan_buffers() {
  const int* dm = d_.dims;
  const int L = d_.num_layers;
  const long B = d_.batch;
  std::vector<size_t> st, ws;   // byte sizes, indexed by buffer id
  auto partial_floats = [](long rows, long cols) { return column_sum_ws_floats(rows, cols); };
  long partial = 0;
  gemm_ws_bytes_ = dt_ ? (64u << 20) : (8u << 20);   // split-K partials
  switch (d_.kind) {
    case SPECTRAIN_KIND_FC: {
      const long C = dm[1], hid = dm[2], maxw = std::max<long>(std::max<long>(dm[0], dm[1]), dm[2]);
      for (int l = 1; l < L; ++l) st.push_back(B * hid * esz_);         // act l at id l-1
      st.push_back(d_.head == SPECTRAIN_HEAD_CE ? B * C * esz_ : 0);     // dlogits at id L-1
      ws = {static_cast<size_t>(B * C * 4), static_cast<size_t>(B * maxw * esz_),
            static_cast<size_t>(B * maxw * esz_), static_cast<size_t>(B * 4)};
      partial = partial_floats(B, maxw);
      break;
    }
    case SPECTRAIN_KIND_CONV3X3: {
      const long P = B * dm[2] * dm[3];
      for (int l = 1; l < L; ++l) st.push_back(P * dm[1] * esz_);
      const bool ce = d_.head == SPECTRAIN_HEAD_CE;
      const long V = ce ? dm[4] : 0;
      st.push_back(ce ? P * dm[1] * esz_ : 0);   // id L-1: last output (the pooled tensor)
      st.push_back(ce ? B * dm[1] * 2 : 0);      // id L: pooled [B, C_out]
      st.push_back(B * V * 2);                   // id L+1: class-score gradient
      const long cmax = std::max(dm[0], dm[1]);
      ws = {static_cast<size_t>(P * cmax * esz_), static_cast<size_t>(P * cmax * esz_),
            static_cast<size_t>(B * V * 4), static_cast<size_t>(ce ? B * 4 : 0),
            static_cast<size_t>(ce ? B * dm[1] * 2 : 0),
            static_cast<size_t>(9L * dm[1] * (dm[0] + (L - 1L) * dm[1]) * esz_)};   // id 5: transposed filters
      partial = partial_floats(B, V);
      for (int l = 0; l < L && dt_; ++l) {   // filter-gradient partials, reduced by the update
        const int C = l == 0 ? dm[0] : dm[1];
        const int sp = std::max(gemm_bf16_split_rule(dm[1], 9 * C, static_cast<int>(P), 1, gemm_ws_bytes_, false),
                                 gemm_bf16_split_rule(dm[1], 9 * C, static_cast<int>(P), 1, gemm_ws_bytes_, true));
        defer_cap_ += static_cast<long>(sp) * dm[1] * 9 * C;
      }
      break;
    }
    case SPECTRAIN_KIND_BOTTLENECK: {
      const long P = B * dm[2] * dm[3], C = dm[0], Cm = dm[1];
      const bool ce = d_.head == SPECTRAIN_HEAD_CE;
      const long V = ce ? dm[4] : 0;
      for (int l = 0; l < L; ++l) {
        st.push_back(P * Cm * esz_);
        st.push_back(P * Cm * esz_);
        st.push_back(l < L - 1 || ce ? P * C * esz_ : 0);
      }
      st.push_back(ce ? B * C * 2 : 0);   // id 3L: pooled [B, C]
      st.push_back(B * V * 2);   // id 3L+1: class-score gradient
      ws = {static_cast<size_t>(P * C * esz_), static_cast<size_t>(P * C * esz_), static_cast<size_t>(P * Cm * esz_),
            static_cast<size_t>(P * Cm * esz_), static_cast<size_t>(B * V * 4), static_cast<size_t>(ce ? B * 4 : 0),
            static_cast<size_t>(ce ? B * C * 2 : 0)};
      partial = partial_floats(B, V);
      break;
    }
    case SPECTRAIN_KIND_TRANSFORMER: {
      const long d = dm[0], H = dm[1], F = dm[2], S = dm[3], T = B * S;
      const bool ce = d_.head == SPECTRAIN_HEAD_CE;
      const long V = ce ? dm[4] : 0;
      const bool fused = attention_fused_supported(static_cast<int>(S), static_cast<int>(d / H), static_cast<int>(d));
      // the fused attention keeps only softmax row statistics; the GEMM path P (f32, bf16) and the scores
      const long BHSS = fused ? 0 : B * H * S * S;
      for (int l = 0; l < L; ++l) {
        size_t s[13] = {static_cast<size_t>(T * 3 * d * 2), static_cast<size_t>(fused ? B * H * S * 2 * 4 : BHSS * 4),
                        static_cast<size_t>(BHSS * 2),      static_cast<size_t>(T * d * 2),
                        static_cast<size_t>(T * d * 2),     static_cast<size_t>(T * 4),
                        static_cast<size_t>(T * 4),         static_cast<size_t>(T * d * 2),
                        static_cast<size_t>(T * F * 2),     static_cast<size_t>(T * d * 2),
                        static_cast<size_t>(T * 4),         static_cast<size_t>(T * 4),
                        static_cast<size_t>(l < L - 1 || ce ? T * d * 2 : 0)};
        st.insert(st.end(), s, s + 13);
      }
      st.push_back(ce ? T * V * 2 : 0);   // dlogits (bf16) at id 13 L
      ws = {static_cast<size_t>(BHSS * 4), static_cast<size_t>(BHSS * 2), static_cast<size_t>(T * d * 2),
            static_cast<size_t>(T * d * 2), static_cast<size_t>(T * d * 2), static_cast<size_t>(T * F * 2),
            static_cast<size_t>(T * d * 2), static_cast<size_t>(T * d * 2), static_cast<size_t>(T * d * 2),
            static_cast<size_t>(T * 3 * d * 2), static_cast<size_t>(ce ? T * V * 4 : 0),
            static_cast<size_t>(ce ? T * 4 : 0)};
      partial = std::max(partial_floats(T, 3 * d), partial_floats(T, F));
      if (ce) partial = std::max(partial, partial_floats(T, V));
      partial = std::max(partial, layernorm_bwd_ws_floats(T, d));
      break;
    }
    case SPECTRAIN_KIND_RESLSTM: {
      const long H = dm[1], T = dm[2], V = dm[3], TB = T * B;
      const bool ce = d_.head == SPECTRAIN_HEAD_CE;
      for (int l = 0; l < L; ++l) {
        st.push_back(TB * 4 * H * 4);
        st.push_back(TB * H * 4);
        st.push_back(TB * H * 2);
        st.push_back((l < L - 1 || ce) ? TB * H * 2 : 0);
      }
      st.push_back(ce ? TB * V * 2 : 0);
      ws = {static_cast<size_t>(TB * 4 * H * 4), static_cast<size_t>(ce ? TB * V * 4 : 0),
            static_cast<size_t>(TB * H * 2),     static_cast<size_t>(TB * H * 2),
            static_cast<size_t>(TB * 4 * H * 2), static_cast<size_t>(B * H * 4),
            static_cast<size_t>(B * H * 4),      static_cast<size_t>(TB * 4),
            static_cast<size_t>(lstm_step_supported(B, static_cast<int>(H)) ? 4 * H * H * 2 : 0)};
      partial = std::max(partial_floats(TB, 4 * H), ce ? partial_floats(TB, V) : 0);
      break;
    }
  }
  ws_colsum_ = static_cast<int>(ws.size());
  ws.push_back(static_cast<size_t>(std::max<long>(partial, 1) * 4));  // column-sum partials, stage stream
  ws_colsum2_ = static_cast<int>(ws.size());
  ws.push_back(static_cast<size_t>(std::max<long>(partial, 1) * 4));  // column-sum partials, side stream
  ws_split_ = static_cast<int>(ws.size());
  ws.push_back(std::max<size_t>(gemm_ws_bytes_, 1));                   // split-K partials, stage stream
  ws_split2_ = static_cast<int>(ws.size());
  ws.push_back(std::max<size_t>(gemm_ws_bytes_, 1));                   // split-K partials, side stream
  if (defer_cap_ > 0) {
    const size_t o = defer_block_.add(static_cast<size_t>(defer_cap_) * 4);
    defer_block_.allocate();
    defer_ = defer_block_.at<float>(o);
  }
  DeviceBlock probe;
  stash_bytes_ = st;
  for (size_t b : st) stash_off_.push_back(probe.add(std::max<size_t>(b, 1)));
  for (size_t b : ws) ws_off_.push_back(ws_block_.add(std::max<size_t>(b, 1)));
  // a second copy for a forward that runs beside a backward (the combined
  // call), allocated here so that the call itself allocates nothing
  for (size_t b : ws) ws_block_f_.add(std::max<size_t>(b, 1));
  const int nslots = d_.num_stages - d_.stage_index;
  slots_.resize(nslots);
  slot_blocks_.resize(nslots);
  for (int i = 0; i < nslots; ++i) {
    for (size_t b : st) slot_blocks_[i].add(std::max<size_t>(b, 1));
    slot_blocks_[i].allocate();
  }
  ws_block_.allocate();
  ws_block_f_.allocate();
}

// ---------------------------------------------------------------- create ----
Stage::Stage(const spectrain_stage_desc& d, const float* W0, size_t n_params, hipStream_t s) : d_(d), s_(s) {
  if (d.abi_version != SPECTRAIN_ABI_VERSION) fail("abi_version mismatch");
  if (d.num_stages < 1 || d.stage_index < 0 || d.stage_index >= d.num_stages) fail("stage_index outside [0, N)");
  if (d.batch < 1 || d.num_layers < 1) fail("batch and num_layers must be >= 1");
  if (!(d.lr > 0.0f) || !std::isfinite(d.lr)) fail("lr must be a positive finite number");
  if (!(d.momentum > 0.0f && d.momentum <= 1.0f)) fail("momentum must lie in (0, 1]");
  if (d.weight_policy != SPECTRAIN_POLICY_PREDICT && d.weight_policy != SPECTRAIN_POLICY_STASH)
    fail("weight_policy must be PREDICT or STASH");
  if (d.dtype != SPECTRAIN_FP32 && d.dtype != SPECTRAIN_BF16) fail("unknown dtype");
  if (d.head != SPECTRAIN_HEAD_NONE && d.head != SPECTRAIN_HEAD_CE) fail("unknown head");
  if (d.head == SPECTRAIN_HEAD_CE && d.kind != SPECTRAIN_KIND_FC && d.kind != SPECTRAIN_KIND_RESLSTM &&
      d.kind != SPECTRAIN_KIND_TRANSFORMER && d.kind != SPECTRAIN_KIND_CONV3X3 && d.kind != SPECTRAIN_KIND_BOTTLENECK)
    fail("unknown stage kind for a CE head");
  dt_ = d.dtype == SPECTRAIN_BF16 ? 1 : 0;
  esz_ = dt_ ? 2 : 4;
  const int* dm = d.dims;
  auto need = [&](int count) {
    for (int i = 0; i < count; ++i)
      if (dm[i] < 1) fail("dims[" + std::to_string(i) + "] must be >= 1");
  };
  auto mult8 = [&](long v, const char* what) {
    if (v % 8) fail(std::string(what) + " must be a multiple of 8 for bf16 stages");
  };
  switch (d.kind) {
    case SPECTRAIN_KIND_FC:
      need(3);
      if (dt_) {
        mult8(dm[0], "in_features");
        mult8(dm[1], "out_features");
        mult8(dm[2], "hidden");
      }
      break;
    case SPECTRAIN_KIND_CONV3X3:
    case SPECTRAIN_KIND_BOTTLENECK:
      need(4);
      if (!dt_) fail("convolution stages run in bf16 only");
      mult8(dm[0], "channels");
      mult8(dm[1], "channels");
      if (d.head == SPECTRAIN_HEAD_CE) {
        need(5);
        if (dm[4] % 2) fail("classes must be even (rows of the class-score gradient are 4-byte aligned)");
      }
      break;
    case SPECTRAIN_KIND_TRANSFORMER:
      need(4);
      if (!dt_) fail("transformer stages run in bf16 only");
      if (dm[0] % dm[1]) fail("d_model must be divisible by heads");
      if (dm[0] % 64 || dm[0] > 2048 || ((dm[0] / 64) & (dm[0] / 64 - 1)))
        fail("d_model must be 64 times a power of two, up to 2048");
      mult8(dm[0] / dm[1], "head dimension");
      mult8(dm[2], "ffn");
      mult8(dm[3], "seq");
      if (d.head == SPECTRAIN_HEAD_CE) {
        need(5);
        mult8(dm[4], "vocab");
      }
      break;
    case SPECTRAIN_KIND_RESLSTM:
      need(3);
      if (!dt_) fail("LSTM stages run in bf16 only");
      if (dm[0] != dm[1]) fail("residual LSTM needs input == hidden");
      mult8(dm[1], "hidden");
      if (d.head == SPECTRAIN_HEAD_CE) {
        need(4);
        mult8(dm[3], "vocab");
      }
      break;
    default:
      fail("unknown stage kind");
  }
  build_layout();
  if (n_params != n_params_) fail("n_params " + std::to_string(n_params) + " != " + std::to_string(n_params_));
  if (!W0) fail("W0_host is NULL");

  hip_check(hipGetDevice(&device_), "hipGetDevice");
  ls_ = s_;
  hip_check(hipStreamCreateWithFlags(&s2_, hipStreamNonBlocking), "hipStreamCreate");
  hip_check(hipEventCreateWithFlags(&fork_ev_, hipEventDisableTiming), "hipEventCreate");
  hip_check(hipEventCreateWithFlags(&join_ev_, hipEventDisableTiming), "hipEventCreate");
  side_ev_.resize(32, nullptr);
  for (hipEvent_t& e : side_ev_) hip_check(hipEventCreateWithFlags(&e, hipEventDisableTiming), "hipEventCreate");
  hip_check(hipStreamCreateWithFlags(&s3_, hipStreamNonBlocking), "hipStreamCreate");
  hip_check(hipEventCreateWithFlags(&ffork_ev_, hipEventDisableTiming), "hipEventCreate");
  hip_check(hipEventCreateWithFlags(&fjoin_ev_, hipEventDisableTiming), "hipEventCreate");
  // arenas: W, v, g (float32), two predicted slots (operand dtype), all padded
  size_t oW = arena_.add(n_arena_ * 4), ov = arena_.add(n_arena_ * 4), og = arena_.add(n_arena_ * 4);
  size_t of = arena_.add(n_arena_ * esz_), ob = arena_.add(n_arena_ * esz_);
  arena_.allocate();
  W_ = arena_.at<float>(oW);
  v_ = arena_.at<float>(ov);
  g_ = arena_.at<float>(og);
  what_[0] = arena_.at<void>(of);
  what_[1] = arena_.at<void>(ob);
  flag_.allocate(1);
  plan_buffers();
  if (d.weight_policy == SPECTRAIN_POLICY_STASH) {
    for (size_t i = 0; i < slots_.size(); ++i) wstash_off_.push_back(wstash_.add(n_arena_ * esz_));
    wstash_.allocate();
  }

  try {
    hip_check(fill_f32(v_, 0.0f, n_arena_, s_), "clear v");
    hip_check(fill_f32(g_, 0.0f, n_arena_, s_), "clear g");
    set_state(W0, nullptr);
  } catch (...) {
    // the member buffers are freed on the way out: let the work already
    // enqueued on them finish first
    (void)hipStreamSynchronize(s_);
    throw;
  }
}

Stage::~Stage() {
  (void)hipStreamSynchronize(s_);
  if (s2_) (void)hipStreamSynchronize(s2_);
  if (s3_) (void)hipStreamSynchronize(s3_);
  for (hipEvent_t e : prof_pool_) (void)hipEventDestroy(e);
  if (fork_ev_) (void)hipEventDestroy(fork_ev_);
  if (join_ev_) (void)hipEventDestroy(join_ev_);
  for (hipEvent_t e : side_ev_)
    if (e) (void)hipEventDestroy(e);
  if (ffork_ev_) (void)hipEventDestroy(ffork_ev_);
  if (fjoin_ev_) (void)hipEventDestroy(fjoin_ev_);
  if (s2_) (void)hipStreamDestroy(s2_);
  if (s3_) (void)hipStreamDestroy(s3_);
}

void Stage::sync() { hip_check(hipStreamSynchronize(s_), "hipStreamSynchronize"); }

// ------------------------------------------------------ state transfer ----
void Stage::set_state(const float* W, const float* v) {
  for (const Slot& sl : slots_)
    if (sl.used) throw StageError(SPECTRAIN_ESTATE, "set_state with mini-batches in flight");
  if (!W) fail("W_host is NULL");
  std::vector<float> hw(n_arena_, 0.0f), hv(n_arena_, 0.0f);
  long src = 0;
  for (const TensorInfo& t : tensors_) {
    std::memcpy(hw.data() + t.off, W + src, t.n * 4);
    if (v) std::memcpy(hv.data() + t.off, v + src, t.n * 4);
    src += t.n;
  }
  hip_check(hipMemcpyAsync(W_, hw.data(), n_arena_ * 4, hipMemcpyHostToDevice, s_), "copy W");
  hip_check(hipMemcpyAsync(v_, hv.data(), n_arena_ * 4, hipMemcpyHostToDevice, s_), "copy v");
  sync();
  predict(0, 0);
  predict(0, 1);
  sync();
  *flag_.host() = 0;
  g_pending_ = false;
}

void Stage::get_state(float* W, float* v) {
  sync();
  std::vector<float> h(n_arena_);
  for (int which = 0; which < 2; ++which) {
    float* dst = which == 0 ? W : v;
    if (!dst) continue;
    hip_check(hipMemcpy(h.data(), which == 0 ? W_ : v_, n_arena_ * 4, hipMemcpyDeviceToHost), "copy state");
    long o = 0;
    for (const TensorInfo& t : tensors_) {
      std::memcpy(dst + o, h.data() + t.off, t.n * 4);
      o += t.n;
    }
  }
}

void Stage::get_predicted(int slot, float* out) {
  if (slot < 0 || slot > 1) fail("slot must be 0 or 1");
  if (!out) fail("What_host is NULL");
  sync();
  std::vector<char> h(n_arena_ * esz_);
  hip_check(hipMemcpy(h.data(), what_[slot], n_arena_ * esz_, hipMemcpyDeviceToHost), "copy predicted");
  long o = 0;
  for (const TensorInfo& t : tensors_) {
    for (long i = 0; i < t.n; ++i) {
      if (dt_) {
        uint32_t bits = static_cast<uint32_t>(reinterpret_cast<const uint16_t*>(h.data())[t.off + i]) << 16;
        std::memcpy(out + o + i, &bits, 4);
      } else {
        out[o + i] = reinterpret_cast<const float*>(h.data())[t.off + i];
      }
    }
    o += t.n;
  }
}

size_t Stage::read_stash(int64_t mb, int index, void* host, size_t capacity) {
  int slot = -1;
  for (size_t i = 0; i < slots_.size(); ++i)
    if (slots_[i].used && slots_[i].mb == mb) slot = static_cast<int>(i);
  if (slot < 0) throw StageError(SPECTRAIN_ESTATE, "mini-batch is not in flight");
  if (index < 0 || static_cast<size_t>(index) >= stash_bytes_.size()) fail("stash index outside the stage's list");
  const size_t n = stash_bytes_[index];
  if (n == 0 || !host) return n;
  if (capacity < n) fail("host buffer of " + std::to_string(capacity) + " bytes is smaller than the stash buffer (" +
                         std::to_string(n) + " bytes)");
  sync();
  hip_check(hipMemcpy(host, slot_blocks_[slot].at<char>(stash_off_[index]), n, hipMemcpyDeviceToHost), "copy stash");
  return n;
}

// --------------------------------------------------- predict and update ----
void Stage::predict(int s, int slot) {
  if (s < 0) fail("version difference must be >= 0");
  if (slot < 0 || slot > 1) fail("slot must be 0 or 1");
  LAUNCH("predict", 0, static_cast<double>(n_params_) * (8 + esz_), predict_slot(W_, v_, what_[slot], dt_, n_arena_, d_.lr, s, s_));
}

void Stage::update(int s_f, int s_b) {
  if (!g_pending_) throw StageError(SPECTRAIN_ESTATE, "update without a gradient from a backward pass");
  // algorithmic: W, v, g read and W, v written (float32), each refreshed slot
  // written in the operand dtype
  const double bytes = static_cast<double>(n_params_) * (12 + 8 + (s_f >= 0) * esz_ + (s_b >= 0) * esz_);
  if (defer_segs_.empty()) {
    LAUNCH("fused_update", 0, bytes,
           fused_update(W_, v_, g_, what_[0], what_[1], dt_, n_arena_, d_.lr, d_.momentum, s_f, s_b, flag_.dev(), s_));
  } else {
    std::sort(defer_segs_.begin(), defer_segs_.end(),
              [](const UpdateSegment& a, const UpdateSegment& b) { return a.off < b.off; });
    double extra = 0.0;   // the partial planes read in place of g: splits - 1 planes more
    for (const UpdateSegment& sg : defer_segs_) extra += 4.0 * (sg.splits - 1) * sg.n;
    LAUNCH_X("fused_update", 0, bytes, extra,
             fused_update_partials(W_, v_, g_, defer_segs_.data(), static_cast<int>(defer_segs_.size()), what_[0],
                                   what_[1], dt_, n_arena_, d_.lr, d_.momentum, s_f, s_b, flag_.dev(), s_));
  }
  defer_segs_.clear();
  defer_used_ = 0;
  g_pending_ = false;
}

// ------------------------------------------------------ forward/backward ----
void Stage::forward(int64_t mb, const void* x, void* y, const int32_t* labels, float* loss) {
  const bool ce = d_.head == SPECTRAIN_HEAD_CE;
  if (!x) fail("x_dev is NULL");
  if (ce && (!labels || !loss)) fail("a CE head needs labels_dev and loss_dev");
  if (!ce && !y) fail("y_dev is NULL");
  int free_slot = -1;
  for (size_t i = 0; i < slots_.size(); ++i) {
    if (slots_[i].used && slots_[i].mb == mb) throw StageError(SPECTRAIN_ESTATE, "mini-batch already in flight");
    if (!slots_[i].used && free_slot < 0) free_slot = static_cast<int>(i);
  }
  if (free_slot < 0) throw StageError(SPECTRAIN_ESTATE, "N - k mini-batches already in flight");
  if (d_.weight_policy == SPECTRAIN_POLICY_STASH)
    hip_check(hipMemcpyAsync(wstash_.at<char>(wstash_off_[free_slot]), what_[0], n_arena_ * esz_,
                             hipMemcpyDeviceToDevice, ls_),
              "stash weights");
  switch (d_.kind) {
    case SPECTRAIN_KIND_FC: fwd_fc(free_slot, x, y, labels, loss); break;
    case SPECTRAIN_KIND_CONV3X3: fwd_conv(free_slot, x, y, labels, loss); break;
    case SPECTRAIN_KIND_BOTTLENECK: fwd_bneck(free_slot, x, y, labels, loss); break;
    case SPECTRAIN_KIND_TRANSFORMER: fwd_tfm(free_slot, x, y, labels, loss); break;
    case SPECTRAIN_KIND_RESLSTM: fwd_lstm(free_slot, x, y, labels, loss); break;
  }
  slots_[free_slot] = Slot{true, mb, x, y};
}

void Stage::backward(int64_t mb, const void* dy, void* dx) {
  int slot = -1;
  for (size_t i = 0; i < slots_.size(); ++i)
    if (slots_[i].used && slots_[i].mb == mb) slot = static_cast<int>(i);
  if (slot < 0) throw StageError(SPECTRAIN_ESTATE, "backward of a mini-batch that is not in flight");
  if (g_pending_) throw StageError(SPECTRAIN_ESTATE, "the previous gradient has not been applied by an update");
  if (d_.head != SPECTRAIN_HEAD_CE && !dy) fail("dy_dev is NULL");
  bwd_weights_ = d_.weight_policy == SPECTRAIN_POLICY_STASH ? wstash_.at<char>(wstash_off_[slot]) : what_[1];
  defer_segs_.clear();
  defer_used_ = 0;
  try {
    switch (d_.kind) {
      case SPECTRAIN_KIND_FC: bwd_fc(slot, dy, dx); break;
      case SPECTRAIN_KIND_CONV3X3: bwd_conv(slot, dy, dx); break;
      case SPECTRAIN_KIND_BOTTLENECK: bwd_bneck(slot, dy, dx); break;
      case SPECTRAIN_KIND_TRANSFORMER: bwd_tfm(slot, dy, dx); break;
      case SPECTRAIN_KIND_RESLSTM: bwd_lstm(slot, dy, dx); break;
    }
  } catch (...) {
    join_side();
    throw;
  }
  join_side();   // the side stream's gradients are complete before anything later on the stage stream
  slots_[slot] = Slot{};
  g_pending_ = true;
}

void Stage::backward_noalloc(int64_t mb, const void* dy, void* dx) {
  if (2 * gemm_ws_bytes_ > SCRATCH_BYTES)
    fail("the stage's two split-K workspaces (" + std::to_string(2 * gemm_ws_bytes_) + " bytes) exceed the " +
         std::to_string(SCRATCH_BYTES) + "-byte scratch of the allocation-free backward");
  float* scratch = device_scratch(device_);
  ext_ws_ = scratch;
  try {
    backward(mb, dy, dx);
  } catch (...) {
    ext_ws_ = nullptr;
    throw;
  }
  ext_ws_ = nullptr;
}

void Stage::forward_backward(int64_t mb_f, const void* x, void* y, const int32_t* labels, float* loss, int64_t mb_b,
                             const void* dy, void* dx) {
  // Every precondition of both passes is checked before anything is issued,
  // so a refused call leaves the stage unchanged.
  const bool ce = d_.head == SPECTRAIN_HEAD_CE;
  if (mb_f == mb_b) throw StageError(SPECTRAIN_ESTATE, "the forward and the backward name the same mini-batch");
  if (!x) fail("x_dev is NULL");
  if (ce && (!labels || !loss)) fail("a CE head needs labels_dev and loss_dev");
  if (!ce && !y) fail("y_dev is NULL");
  if (!ce && !dy) fail("dy_dev is NULL");
  bool b_in_flight = false, has_free = false;
  for (const Slot& sl : slots_) {
    if (sl.used && sl.mb == mb_f) throw StageError(SPECTRAIN_ESTATE, "mini-batch already in flight");
    if (sl.used && sl.mb == mb_b) b_in_flight = true;
    if (!sl.used) has_free = true;
  }
  if (!b_in_flight) throw StageError(SPECTRAIN_ESTATE, "backward of a mini-batch that is not in flight");
  if (!has_free) throw StageError(SPECTRAIN_ESTATE, "N - k mini-batches already in flight");
  if (g_pending_) throw StageError(SPECTRAIN_ESTATE, "the previous gradient has not been applied by an update");
  // the forward starts after everything issued on the stage stream so far
  // (the update that refreshed its weights)
  hip_check(hipEventRecord(ffork_ev_, s_), "hipEventRecord");
  hip_check(hipStreamWaitEvent(s3_, ffork_ev_, 0), "hipStreamWaitEvent");
  ls_ = serial_ ? s_ : s3_;
  wsb_ = &ws_block_f_;
  concurrent_ = true;
  try {
    forward(mb_f, x, y, labels, loss);
  } catch (...) {
    ls_ = s_;
    wsb_ = &ws_block_;
    concurrent_ = false;
    hip_check(hipEventRecord(fjoin_ev_, s3_), "hipEventRecord");
    hip_check(hipStreamWaitEvent(s_, fjoin_ev_, 0), "hipStreamWaitEvent");
    throw;
  }
  ls_ = s_;
  wsb_ = &ws_block_;
  hip_check(hipEventRecord(fjoin_ev_, s3_), "hipEventRecord");
  try {
    backward(mb_b, dy, dx);
  } catch (...) {
    concurrent_ = false;
    hip_check(hipStreamWaitEvent(s_, fjoin_ev_, 0), "hipStreamWaitEvent");
    throw;
  }
  concurrent_ = false;
  hip_check(hipStreamWaitEvent(s_, fjoin_ev_, 0), "hipStreamWaitEvent");
}

// ==================================================================== FC ====
// y_l = relu(a_l W_l^T + b_l); the last layer of a CE stage produces logits.
void Stage::fwd_fc(int slot, const void* x, void* y, const int32_t* labels, float* loss) {
  const int L = d_.num_layers, B = d_.batch;
  const bool ce = d_.head == SPECTRAIN_HEAD_CE;
  const void* a = x;
  for (int l = 0; l < L; ++l) {
    const int fin = l == 0 ? d_.dims[0] : d_.dims[2];
    const int fout = l == L - 1 ? d_.dims[1] : d_.dims[2];
    GemmDesc g = gd(B, fout, fin, opK(a, fin), opK(wf(2 * l), fin), fout);
    if (dt_) g.epi.bias_bf16 = static_cast<const bf16_t*>(wf(2 * l + 1));
    else g.epi.bias = static_cast<const float*>(wf(2 * l + 1));
    void* out;
    if (l == L - 1 && ce) {
      out = ws<float>(0);
      g.epi.out_f32 = static_cast<float*>(out);
    } else {
      out = l == L - 1 ? y : stash<char>(slot, l);
      g.epi.relu = 1;
      if (dt_) g.epi.out_bf16 = static_cast<bf16_t*>(out);
      else g.epi.out_f32 = static_cast<float*>(out);
    }
    gemm(g);
    a = out;
  }
  if (ce)
    LAUNCH("softmax_ce", 0, ce_bytes(B, d_.dims[1]),
           softmax_ce(ws<float>(0), labels, B, d_.dims[1], stash<void>(slot, L - 1), dt_, loss, ws<float>(3), ls_));
}

void Stage::bwd_fc(int slot, const void* dy, void* dx) {
  const int L = d_.num_layers, B = d_.batch;
  const Slot& sl = slots_[slot];
  auto act = [&](int l) -> const void* { return l == 0 ? sl.x : (l == L ? sl.y : stash<char>(slot, l - 1)); };
  auto width = [&](int l) { return l == 0 ? d_.dims[0] : (l == L ? d_.dims[1] : d_.dims[2]); };
  const void* dz;
  if (d_.head == SPECTRAIN_HEAD_CE) {
    dz = stash<void>(slot, L - 1);
  } else {
    LAUNCH("mask", 0, 3.0 * esz_ * B * d_.dims[1],
           mask_relu_grad(dy, sl.y, ws<void>(1), static_cast<long>(B) * d_.dims[1], dt_, s_));
    dz = ws<void>(1);
  }
  int pp = 2;
  for (int l = L - 1; l >= 0; --l) {
    const int fin = width(l), fout = width(l + 1);
    GemmDesc gw = gd(fout, fin, B, opR(dz, fout), opR(act(l), fin), fin);
    gw.epi.out_f32 = grad(2 * l);
    gemm(gw);
    LAUNCH("bias_grad", 0, colsum_bytes(B, fout, esz_), column_sum(dz, dt_, B, fout, fout, grad(2 * l + 1), 0, ws<float>(ws_colsum_), s_));
    if (l == 0 && !dx) break;
    void* out = l == 0 ? dx : ws<void>(pp);
    GemmDesc gx = gd(B, fin, fout, opK(dz, fout), opR(wb(2 * l), fin), fin);
    if (dt_) gx.epi.out_bf16 = static_cast<bf16_t*>(out);
    else gx.epi.out_f32 = static_cast<float*>(out);
    if (l > 0) gx.epi.mask = act(l);
    gemm(gx);
    dz = out;
    pp = pp == 2 ? 1 : 2;
  }
}

// ========================================================== CONV 3x3 ====
// stash ids: l - 1 the output of layer l - 1 (input of layer l, l >= 1); with a
// CE head also L - 1 the last output, L the pooled tensor, L + 1 the
// class-score gradient. workspace: 0/1 gradient ping-pong, 2 class scores
// (f32), 3 per-sample losses, 4 pooled gradient, then column-sum partials.
void Stage::fwd_conv(int slot, const void* x, void* y, const int32_t* labels, float* loss) {
  const int L = d_.num_layers, B = d_.batch, Cin = d_.dims[0], Cout = d_.dims[1], H = d_.dims[2], W = d_.dims[3];
  const int P = B * H * W;
  const bool ce = d_.head == SPECTRAIN_HEAD_CE;
  const void* a = x;
  for (int l = 0; l < L; ++l) {
    const int C = l == 0 ? Cin : Cout;
    void* out = l == L - 1 && !ce ? y : stash<void>(slot, l);
    GemmDesc g = gd(P, Cout, 9 * C, opConv(OP_K_CONV_FWD, a, B, H, W, C), opK(wf(l), 9 * C), Cout);
    g.epi.relu = 1;
    g.epi.out_bf16 = static_cast<bf16_t*>(out);
    gemm(g);
    a = out;
  }
  if (ce) pool_head_fwd(slot, a, H * W, Cout, L, L, L + 1, 2, labels, loss);
}

// Classifier of a conv stage with a CE head (global average pool over H x W,
// linear to the classes, mean softmax cross-entropy over the batch). yl is the
// stage's last output [B, HW, C]; tensor t is the classifier weight (t + 1 its
// bias); the pooled tensor and the class-score gradient go to stash ids
// id_pool, id_dl; workspace ids wsl, wsl + 1, wsl + 2 hold the float32 scores,
// the per-sample losses and the pooled gradient.
void Stage::pool_head_fwd(int slot, const void* yl, int HW, int C, int t, int id_pool, int id_dl, int wsl,
                          const int32_t* labels, float* loss) {
  const int B = d_.batch, V = d_.dims[4];
  bf16_t* pooled = stash<bf16_t>(slot, id_pool);
  LAUNCH("avgpool", 0, 2.0 * B * C * (HW + 1),
         avgpool_fwd(static_cast<const bf16_t*>(yl), B, HW, C, pooled, ls_));
  GemmDesc g = gd(B, V, C, opK(pooled, C), opK(wf(t), C), V);
  g.epi.bias_bf16 = static_cast<const bf16_t*>(wf(t + 1));
  g.epi.out_f32 = ws<float>(wsl);
  gemm(g);
  LAUNCH("softmax_ce", 0, ce_bytes(B, V), softmax_ce(ws<float>(wsl), labels, B, V, stash<void>(slot, id_dl), 1, loss,
                                        ws<float>(wsl + 1), ls_));
}

void Stage::pool_head_bwd(int slot, const void* yl, int HW, int C, int t, int id_pool, int id_dl, int wsl, void* dz) {
  const int B = d_.batch, V = d_.dims[4];
  const bf16_t* dl = stash<bf16_t>(slot, id_dl);
  const bf16_t* pooled = stash<bf16_t>(slot, id_pool);
  GemmDesc gw = gd(V, C, B, opR(dl, V), opR(pooled, C), C);
  gw.epi.out_f32 = grad(t);
  gemm(gw);
  LAUNCH("bias_grad", 0, colsum_bytes(B, V, 2),
         column_sum(dl, 1, B, V, V, grad(t + 1), 0, ws<float>(ws_colsum_), s_));
  bf16_t* dpool = ws<bf16_t>(wsl + 2);
  GemmDesc gx = gd(B, C, V, opK(dl, V), opR(wb(t), C), C);
  gx.epi.out_bf16 = dpool;
  gemm(gx);
  LAUNCH("avgpool_bwd", 0, 2.0 * B * C * (2 * HW + 1),
         avgpool_bwd_mask(dpool, static_cast<const bf16_t*>(yl), B, HW, C, static_cast<bf16_t*>(dz), s_));
}

void Stage::bwd_conv(int slot, const void* dy, void* dx) {
  const int L = d_.num_layers, B = d_.batch, Cin = d_.dims[0], Cout = d_.dims[1], H = d_.dims[2], W = d_.dims[3];
  const int P = B * H * W;
  const Slot& sl = slots_[slot];
  auto act = [&](int l) -> const void* { return l == 0 ? sl.x : stash<void>(slot, l - 1); };
  if (d_.head == SPECTRAIN_HEAD_CE)
    pool_head_bwd(slot, stash<void>(slot, L - 1), H * W, Cout, L, L, L + 1, 2, ws<void>(0));
  else
    LAUNCH("mask", 0, 6.0 * P * Cout, mask_relu_grad(dy, sl.y, ws<void>(0), static_cast<long>(P) * Cout, 1, s_));
  const void* dz = ws<void>(0);
  // the data gradients read each filter transposed ([C][9][C_out], k
  // contiguous), made for every layer that needs one in launches of up to
  // FilterBatch::MAX layers
  std::vector<bf16_t*> wt(L);
  {
    bf16_t* p = ws<bf16_t>(5);
    for (int l = 0; l < L; ++l) {
      wt[l] = p;
      p += 9L * Cout * (l == 0 ? Cin : Cout);
    }
    FilterBatch fb{};
    fb.Co = Cout;
    double bytes = 0;
    for (int l = dx ? 0 : 1; l < L; ++l) {
      fb.W[fb.n] = static_cast<const bf16_t*>(wb(l));
      fb.Wt[fb.n] = wt[l];
      fb.Ci[fb.n] = l == 0 ? Cin : Cout;
      bytes += 4.0 * 9 * Cout * fb.Ci[fb.n];
      if (++fb.n == FilterBatch::MAX || l == L - 1) {
        LAUNCH("filter_transpose", 0, bytes, filter_transpose_bf16(fb, s_));
        fb.n = 0;
        bytes = 0;
      }
    }
  }
  int pp = 1;
  for (int l = L - 1; l >= 0; --l) {
    const int C = l == 0 ? Cin : Cout;
    GemmDesc gw = gd(Cout, 9 * C, P, opR(dz, Cout), opConv(OP_R_CONV_WGRAD, act(l), B, H, W, C), 9 * C);
    gw.epi.out_f32 = grad(l);
    gemm(gw, true);
    if (l == 0 && !dx) break;
    void* out = l == 0 ? dx : ws<void>(pp);
    GemmDesc gx = gd(P, C, 9 * Cout, opConv(OP_K_CONV_DGRAD, dz, B, H, W, Cout), opK(wt[l], 9 * Cout), C);
    gx.epi.out_bf16 = static_cast<bf16_t*>(out);
    if (l > 0) gx.epi.mask = act(l);
    gemm(gx);
    dz = out;
    pp ^= 1;
  }
}

// ======================================================== BOTTLENECK ====
// y = relu(x + conv1x1_3(relu(conv3x3_2(relu(conv1x1_1(x)))))).
// stash ids 3 l + j: 0 t1, 1 t2, 2 block output (l < L - 1, or every block with
// a CE head); with a CE head 3 L the pooled tensor, 3 L + 1 the class-score
// gradient. workspace: 0/1 output-gradient ping-pong, 2 dt2, 3 dt1, 4 class
// scores (f32), 5 per-sample losses, 6 pooled gradient, then column-sum partials.
void Stage::fwd_bneck(int slot, const void* x, void* y, const int32_t* labels, float* loss) {
  const int L = d_.num_layers, B = d_.batch, C = d_.dims[0], Cm = d_.dims[1], H = d_.dims[2], W = d_.dims[3];
  const int P = B * H * W;
  const bool ce = d_.head == SPECTRAIN_HEAD_CE;
  const void* a = x;
  for (int l = 0; l < L; ++l) {
    bf16_t* t1 = stash<bf16_t>(slot, 3 * l);
    bf16_t* t2 = stash<bf16_t>(slot, 3 * l + 1);
    void* out = l == L - 1 && !ce ? y : stash<void>(slot, 3 * l + 2);
    GemmDesc g1 = gd(P, Cm, C, opK(a, C), opK(wf(3 * l), C), Cm);
    g1.epi.relu = 1;
    g1.epi.out_bf16 = t1;
    gemm(g1);
    GemmDesc g2 = gd(P, Cm, 9 * Cm, opConv(OP_K_CONV_FWD, t1, B, H, W, Cm), opK(wf(3 * l + 1), 9 * Cm), Cm);
    g2.epi.relu = 1;
    g2.epi.out_bf16 = t2;
    gemm(g2);
    GemmDesc g3 = gd(P, C, Cm, opK(t2, Cm), opK(wf(3 * l + 2), Cm), C);
    g3.epi.relu = 1;
    g3.epi.res_bf16 = static_cast<const bf16_t*>(a);
    g3.epi.out_bf16 = static_cast<bf16_t*>(out);
    gemm(g3);
    a = out;
  }
  if (ce) pool_head_fwd(slot, a, H * W, C, 3 * L, 3 * L, 3 * L + 1, 4, labels, loss);
}

void Stage::bwd_bneck(int slot, const void* dy, void* dx) {
  const int L = d_.num_layers, B = d_.batch, C = d_.dims[0], Cm = d_.dims[1], H = d_.dims[2], W = d_.dims[3];
  const int P = B * H * W;
  const Slot& sl = slots_[slot];
  auto xin = [&](int l) -> const void* { return l == 0 ? sl.x : stash<void>(slot, 3 * (l - 1) + 2); };
  // dr: gradient at the block's pre-ReLU output (after the output mask)
  if (d_.head == SPECTRAIN_HEAD_CE)
    pool_head_bwd(slot, stash<void>(slot, 3 * (L - 1) + 2), H * W, C, 3 * L, 3 * L, 3 * L + 1, 4, ws<void>(0));
  else
    LAUNCH("mask", 0, 6.0 * P * C, mask_relu_grad(dy, sl.y, ws<void>(0), static_cast<long>(P) * C, 1, s_));
  // The data gradients (d3, d2, d1) form the chain on the stage stream; each
  // weight gradient (g3, g2, g1, with its split-K reduction) runs on the side
  // stream as soon as its input is produced. Before the chain rewrites a
  // workspace buffer (the next block's dt2, dt1, or the dr two blocks back)
  // it waits for the side GEMM that reads it.
  int cur = 0;
  bf16_t* dt2 = ws<bf16_t>(2);
  bf16_t* dt1 = ws<bf16_t>(3);
  for (int l = L - 1; l >= 0; --l) {
    const bf16_t* dr = ws<bf16_t>(cur);
    const bf16_t* t1 = stash<bf16_t>(slot, 3 * l);
    const bf16_t* t2 = stash<bf16_t>(slot, 3 * l + 1);
    GemmDesc g3 = gd(C, Cm, P, opR(dr, C), opR(t2, Cm), Cm);
    g3.epi.out_f32 = grad(3 * l + 2);
    side_gemm(g3, {dr});
    GemmDesc d3 = gd(P, Cm, C, opK(dr, C), opR(wb(3 * l + 2), Cm), Cm);
    d3.epi.out_bf16 = dt2;
    d3.epi.mask = t2;
    protect(dt2);
    gemm(d3);
    GemmDesc g2 = gd(Cm, 9 * Cm, P, opR(dt2, Cm), opConv(OP_R_CONV_WGRAD, t1, B, H, W, Cm), 9 * Cm);
    g2.epi.out_f32 = grad(3 * l + 1);
    side_gemm(g2, {dt2});
    GemmDesc d2 = gd(P, Cm, 9 * Cm, opConv(OP_K_CONV_DGRAD, dt2, B, H, W, Cm),
                     opConv(OP_R_FILTER_T, wb(3 * l + 1), B, H, W, Cm, Cm), Cm);
    d2.epi.out_bf16 = dt1;
    d2.epi.mask = t1;
    protect(dt1);
    gemm(d2);
    GemmDesc g1 = gd(Cm, C, P, opR(dt1, Cm), opR(xin(l), C), C);
    g1.epi.out_f32 = grad(3 * l);
    side_gemm(g1, {dt1});
    if (l == 0 && !dx) break;
    void* out = l == 0 ? dx : ws<void>(cur ^ 1);
    protect(out);
    GemmDesc d1 = gd(P, C, Cm, opK(dt1, Cm), opR(wb(3 * l), C), C);
    d1.epi.res_bf16 = dr;
    d1.epi.out_bf16 = static_cast<bf16_t*>(out);
    if (l > 0) d1.epi.mask = xin(l);
    gemm(d1);
    cur ^= 1;
  }
}

// ======================================================= TRANSFORMER ====
// Post-LN encoder layer; per layer stash ids 13*l + j:
// 0 qkv, 1 P (f32; with the fused attention core the softmax row statistics),
// 2 P (bf16; unused with the fused core), 3 ctx, 4 r1, 5 mean1, 6 rstd1, 7 h,
// 8 f1, 9 r2, 10 mean2, 11 rstd2, 12 layer output (l < L-1, or every layer
// with a CE head); id 13 L: dlogits (bf16) with a CE head.
void Stage::fwd_tfm(int slot, const void* x, void* y, const int32_t* labels, float* loss) {
  const int L = d_.num_layers, B = d_.batch, d = d_.dims[0], Hh = d_.dims[1], F = d_.dims[2], S = d_.dims[3];
  const int T = B * S, dh = d / Hh;
  const bool ce = d_.head == SPECTRAIN_HEAD_CE;
  const float scale = 1.0f / std::sqrt(static_cast<float>(dh));
  const void* a = x;
  for (int l = 0; l < L; ++l) {
    const int p = 12 * l, q = 13 * l;
    bf16_t* qkv = stash<bf16_t>(slot, q);
    float* P = stash<float>(slot, q + 1);
    bf16_t* Pb = stash<bf16_t>(slot, q + 2);
    bf16_t* ctx = stash<bf16_t>(slot, q + 3);
    bf16_t* r1 = stash<bf16_t>(slot, q + 4);
    bf16_t* h = stash<bf16_t>(slot, q + 7);
    bf16_t* f1 = stash<bf16_t>(slot, q + 8);
    bf16_t* r2 = stash<bf16_t>(slot, q + 9);
    void* out = l == L - 1 && !ce ? y : stash<void>(slot, q + 12);

    GemmDesc g = gd(T, 3 * d, d, opK(a, d), opK(wf(p), d), 3 * d);
    g.epi.bias_bf16 = static_cast<const bf16_t*>(wf(p + 1));
    g.epi.out_bf16 = qkv;
    gemm(g);
    if (attention_fused_supported(S, dh, d)) {
      LAUNCH("attention", 4.0 * B * Hh * S * S * dh, 2.0 * T * 4 * d + 8.0 * B * Hh * S,
             attention_fwd(qkv, B, Hh, d, scale, P, ctx, ls_));
    } else {
    // scores[b, h] = Q K^T * scale
    Operand qa = opK(qkv, 3 * d), kb = opK(qkv + d, 3 * d);
    qa.bs1 = kb.bs1 = static_cast<long>(S) * 3 * d;
    qa.bs2 = kb.bs2 = dh;
    GemmDesc sc = gd(S, S, dh, qa, kb, S);
    sc.batch = B * Hh;
    sc.zdiv = Hh;
    sc.epi.bs1 = static_cast<long>(Hh) * S * S;
    sc.epi.bs2 = static_cast<long>(S) * S;
    sc.epi.alpha = scale;
    sc.epi.out_f32 = ws<float>(0);
    gemm(sc);
    LAUNCH("softmax", 0, 10.0 * B * Hh * S * S, softmax_rows(ws<float>(0), B * Hh * S, S, P, Pb, ls_));
    // ctx[b, :, h] = P V
    Operand pa = opK(Pb, S), vb = opR(qkv + 2 * d, 3 * d);
    pa.bs1 = static_cast<long>(Hh) * S * S;
    pa.bs2 = static_cast<long>(S) * S;
    vb.bs1 = static_cast<long>(S) * 3 * d;
    vb.bs2 = dh;
    GemmDesc pv = gd(S, dh, S, pa, vb, d);
    pv.batch = B * Hh;
    pv.zdiv = Hh;
    pv.epi.bs1 = static_cast<long>(S) * d;
    pv.epi.bs2 = dh;
    pv.epi.out_bf16 = ctx;
    gemm(pv);
    }
    GemmDesc go = gd(T, d, d, opK(ctx, d), opK(wf(p + 2), d), d);
    go.epi.bias_bf16 = static_cast<const bf16_t*>(wf(p + 3));
    go.epi.res_bf16 = static_cast<const bf16_t*>(a);
    go.epi.out_bf16 = r1;
    gemm(go);
    LAUNCH("layernorm", 0, ln_bytes(T, d), layernorm_fwd(r1, static_cast<const bf16_t*>(wf(p + 4)), static_cast<const bf16_t*>(wf(p + 5)), T, d,
                            LN_EPS, h, stash<float>(slot, q + 5), stash<float>(slot, q + 6), ls_));
    GemmDesc g1 = gd(T, F, d, opK(h, d), opK(wf(p + 6), d), F);
    g1.epi.bias_bf16 = static_cast<const bf16_t*>(wf(p + 7));
    g1.epi.relu = 1;
    g1.epi.out_bf16 = f1;
    gemm(g1);
    GemmDesc g2 = gd(T, d, F, opK(f1, F), opK(wf(p + 8), F), d);
    g2.epi.bias_bf16 = static_cast<const bf16_t*>(wf(p + 9));
    g2.epi.res_bf16 = h;
    g2.epi.out_bf16 = r2;
    gemm(g2);
    LAUNCH("layernorm", 0, ln_bytes(T, d), layernorm_fwd(r2, static_cast<const bf16_t*>(wf(p + 10)), static_cast<const bf16_t*>(wf(p + 11)), T, d,
                            LN_EPS, static_cast<bf16_t*>(out), stash<float>(slot, q + 10), stash<float>(slot, q + 11),
                            ls_));
    a = out;
  }
  if (ce) {   // logits of every token (float32), mean token cross-entropy, dlogits (bf16) for the backward
    const int V = d_.dims[4];
    GemmDesc gv = gd(T, V, d, opK(a, d), opK(wf(12 * L), d), V);
    gv.epi.bias_bf16 = static_cast<const bf16_t*>(wf(12 * L + 1));
    gv.epi.out_f32 = ws<float>(10);
    gemm(gv);
    LAUNCH("softmax_ce", 0, ce_bytes(T, V), softmax_ce(ws<float>(10), labels, T, V, stash<void>(slot, 13 * L), 1, loss,
                                          ws<float>(11), ls_));
  }
}

// workspace ids: 0 scores/dP (f32), 1 dS, 2/3 layer-output gradient ping-pong,
// 4 dr2, 5 df1, 6 dh, 7 dr1, 8 dctx, 9 dqkv, 10 logits (f32, CE head),
// 11 per-token losses (CE head), 12 column-sum partials
void Stage::bwd_tfm(int slot, const void* dy, void* dx) {
  const int L = d_.num_layers, B = d_.batch, d = d_.dims[0], Hh = d_.dims[1], F = d_.dims[2], S = d_.dims[3];
  const int T = B * S, dh = d / Hh;
  const float scale = 1.0f / std::sqrt(static_cast<float>(dh));
  const Slot& sl = slots_[slot];
  float* part = ws<float>(ws_colsum_);
  float* part2 = ws<float>(ws_colsum2_);
  const void* gy = dy;
  int pp = 2;
  if (d_.head == SPECTRAIN_HEAD_CE) {   // vocabulary head: its gradients and dY of the last layer
    const int V = d_.dims[4];
    const bf16_t* dl = stash<bf16_t>(slot, 13 * L);
    const void* yL = stash<void>(slot, 13 * (L - 1) + 12);
    GemmDesc gw = gd(V, d, T, opR(dl, V), opR(yL, d), d);
    gw.epi.out_f32 = grad(12 * L);
    gemm(gw);
    LAUNCH("bias_grad", 0, colsum_bytes(T, V, 2), column_sum(dl, 1, T, V, V, grad(12 * L + 1), 0, part, s_));
    GemmDesc gx = gd(T, d, V, opK(dl, V), opR(wb(12 * L), d), d);
    gx.epi.out_bf16 = ws<bf16_t>(2);
    gemm(gx);
    gy = ws<void>(2);
    pp = 3;
  }
  for (int l = L - 1; l >= 0; --l) {
    const int p = 12 * l, q = 13 * l;
    const void* a = l == 0 ? sl.x : stash<void>(slot, 13 * (l - 1) + 12);
    const bf16_t* qkv = stash<bf16_t>(slot, q);
    const float* P = stash<float>(slot, q + 1);
    const bf16_t* Pb = stash<bf16_t>(slot, q + 2);
    const bf16_t* ctx = stash<bf16_t>(slot, q + 3);
    const bf16_t* r1 = stash<bf16_t>(slot, q + 4);
    const bf16_t* h = stash<bf16_t>(slot, q + 7);
    const bf16_t* f1 = stash<bf16_t>(slot, q + 8);
    const bf16_t* r2 = stash<bf16_t>(slot, q + 9);
    bf16_t* dr2 = ws<bf16_t>(4);
    bf16_t* df1 = ws<bf16_t>(5);
    bf16_t* dhh = ws<bf16_t>(6);
    bf16_t* dr1 = ws<bf16_t>(7);
    bf16_t* dctx = ws<bf16_t>(8);
    bf16_t* dqkv = ws<bf16_t>(9);

    // layer-norm backward rows on the stage stream; its parameter gradients
    // (and the FFN output bias gradient: column sums of dr2) reduced from the
    // per-block partials on the side stream
    protect(dr2);
    protect(part);
    LAUNCH("layernorm_bwd", 0, lnb_rows_bytes(T, d),
           layernorm_bwd_rows(static_cast<const bf16_t*>(gy), r2, stash<float>(slot, q + 10), stash<float>(slot, q + 11),
                              static_cast<const bf16_t*>(wb(p + 10)), T, d, dr2, part, s_));
    on_side({part}, [&]() {
      LAUNCH("layernorm_bwd_params", 0, lnb_params_bytes(T, d),
             layernorm_bwd_params(part, T, d, grad(p + 10), grad(p + 11), grad(p + 9), ls_));
    });
    GemmDesc w2 = gd(d, F, T, opR(dr2, d), opR(f1, F), F);
    w2.epi.out_f32 = grad(p + 8);
    side_gemm(w2, {dr2});
    GemmDesc x2 = gd(T, F, d, opK(dr2, d), opR(wb(p + 8), F), F);
    x2.epi.mask = f1;
    x2.epi.out_bf16 = df1;
    protect(df1);
    gemm(x2);
    GemmDesc w1 = gd(F, d, T, opR(df1, F), opR(h, d), d);
    w1.epi.out_f32 = grad(p + 6);
    side_gemm(w1, {df1});
    on_side({df1}, [&]() {
      LAUNCH("bias_grad", 0, colsum_bytes(T, F, 2), column_sum(df1, 1, T, F, F, grad(p + 7), 0, part2, ls_));
    });
    GemmDesc x1 = gd(T, d, F, opK(df1, F), opR(wb(p + 6), d), d);
    x1.epi.res_bf16 = dr2;
    x1.epi.out_bf16 = dhh;
    gemm(x1);
    protect(dr1);
    protect(part);
    LAUNCH("layernorm_bwd", 0, lnb_rows_bytes(T, d),
           layernorm_bwd_rows(dhh, r1, stash<float>(slot, q + 5), stash<float>(slot, q + 6),
                              static_cast<const bf16_t*>(wb(p + 4)), T, d, dr1, part, s_));
    on_side({part}, [&]() {   // also the attention output bias gradient: column sums of dr1
      LAUNCH("layernorm_bwd_params", 0, lnb_params_bytes(T, d),
             layernorm_bwd_params(part, T, d, grad(p + 4), grad(p + 5), grad(p + 3), ls_));
    });
    GemmDesc wo = gd(d, d, T, opR(dr1, d), opR(ctx, d), d);
    wo.epi.out_f32 = grad(p + 2);
    side_gemm(wo, {dr1});
    GemmDesc xo = gd(T, d, d, opK(dr1, d), opR(wb(p + 2), d), d);
    xo.epi.out_bf16 = dctx;
    gemm(xo);

    // attention backward: fused, or batched GEMMs over (b, h)
    protect(dqkv);
    if (attention_fused_supported(S, dh, d)) {
      LAUNCH("attention_bwd", 10.0 * B * Hh * S * S * dh, 2.0 * T * 7 * d + 8.0 * B * Hh * S,
             attention_bwd(qkv, dctx, P, B, Hh, d, scale, dqkv, s_));
    } else {
    const long sS = static_cast<long>(S) * S, sHSS = static_cast<long>(Hh) * S * S;
    const long sQ = static_cast<long>(S) * 3 * d, sO = static_cast<long>(S) * d;
    {  // dV = P^T dO
      Operand A = opR(Pb, S), Bo = opR(dctx, d);
      A.bs1 = sHSS;
      A.bs2 = sS;
      Bo.bs1 = sO;
      Bo.bs2 = dh;
      GemmDesc g = gd(S, dh, S, A, Bo, 3 * d);
      g.batch = B * Hh;
      g.zdiv = Hh;
      g.epi.bs1 = sQ;
      g.epi.bs2 = dh;
      g.epi.out_bf16 = dqkv + 2 * d;
      gemm(g);
    }
    {  // dP = dO V^T
      Operand A = opK(dctx, d), Bv = opK(qkv + 2 * d, 3 * d);
      A.bs1 = sO;
      A.bs2 = dh;
      Bv.bs1 = sQ;
      Bv.bs2 = dh;
      GemmDesc g = gd(S, S, dh, A, Bv, S);
      g.batch = B * Hh;
      g.zdiv = Hh;
      g.epi.bs1 = sHSS;
      g.epi.bs2 = sS;
      g.epi.out_f32 = ws<float>(0);
      gemm(g);
    }
    LAUNCH("softmax_bwd", 0, 10.0 * B * Hh * S * S, softmax_bwd(P, ws<float>(0), B * Hh * S, S, ws<bf16_t>(1), s_));
    {  // dQ = dS K * scale
      Operand A = opK(ws<bf16_t>(1), S), Bk = opR(qkv + d, 3 * d);
      A.bs1 = sHSS;
      A.bs2 = sS;
      Bk.bs1 = sQ;
      Bk.bs2 = dh;
      GemmDesc g = gd(S, dh, S, A, Bk, 3 * d);
      g.batch = B * Hh;
      g.zdiv = Hh;
      g.epi.bs1 = sQ;
      g.epi.bs2 = dh;
      g.epi.alpha = scale;
      g.epi.out_bf16 = dqkv;
      gemm(g);
    }
    {  // dK = dS^T Q * scale
      Operand A = opR(ws<bf16_t>(1), S), Bq = opR(qkv, 3 * d);
      A.bs1 = sHSS;
      A.bs2 = sS;
      Bq.bs1 = sQ;
      Bq.bs2 = dh;
      GemmDesc g = gd(S, dh, S, A, Bq, 3 * d);
      g.batch = B * Hh;
      g.zdiv = Hh;
      g.epi.bs1 = sQ;
      g.epi.bs2 = dh;
      g.epi.alpha = scale;
      g.epi.out_bf16 = dqkv + d;
      gemm(g);
    }
    }
    GemmDesc wq = gd(3 * d, d, T, opR(dqkv, 3 * d), opR(a, d), d);
    wq.epi.out_f32 = grad(p);
    side_gemm(wq, {dqkv, a});
    on_side({dqkv}, [&]() {
      LAUNCH("bias_grad", 0, colsum_bytes(T, 3 * d, 2),
             column_sum(dqkv, 1, T, 3 * d, 3 * d, grad(p + 1), 0, part2, ls_));
    });
    if (l == 0 && !dx) break;
    void* out = l == 0 ? dx : ws<void>(pp);
    protect(out);
    GemmDesc xq = gd(T, d, 3 * d, opK(dqkv, 3 * d), opR(wb(p), d), d);
    xq.epi.res_bf16 = dr1;
    xq.epi.out_bf16 = static_cast<bf16_t*>(out);
    gemm(xq);
    gy = out;
    pp = pp == 2 ? 3 : 2;
  }
}

// ===================================================== RESIDUAL LSTM ====
// per layer stash ids 4*l + j: 0 gates (f32 [T,B,4H]), 1 c (f32), 2 h (bf16),
// 3 layer output u_{l+1} (bf16); id 4L: dlogits (bf16) with a CE head.
// workspace: 0 zx (f32), 1 logits (f32), 2/3 du ping-pong, 4 dz (bf16),
// 5 dh_rec (f32), 6 dc (f32), 7 row losses, 8 W_h^T (bf16, fused steps),
// 9 partials. With B <= 64 and H a multiple of 32 every recurrent step is one
// fused launch (contraction + cell); otherwise a GEMM and a cell launch.
void Stage::fwd_lstm(int slot, const void* x, void* y, const int32_t* labels, float* loss) {
  const int L = d_.num_layers, B = d_.batch, I = d_.dims[0], H = d_.dims[1], T = d_.dims[2], V = d_.dims[3];
  const bool ce = d_.head == SPECTRAIN_HEAD_CE;
  const long TB = static_cast<long>(T) * B;
  const void* u = x;
  float* zx = ws<float>(0);
  for (int l = 0; l < L; ++l) {
    const int p = 3 * l, q = 4 * l;
    const int in = l == 0 ? I : H;
    float* gates = stash<float>(slot, q);
    float* c = stash<float>(slot, q + 1);
    bf16_t* hs = stash<bf16_t>(slot, q + 2);
    void* out = (l == L - 1 && !ce) ? y : stash<void>(slot, q + 3);
    GemmDesc gx = gd(static_cast<int>(TB), 4 * H, in, opK(u, in), opK(wf(p), in), 4 * H);
    gx.epi.bias_bf16 = static_cast<const bf16_t*>(wf(p + 2));
    gx.epi.out_f32 = zx;
    gemm(gx);
    const bool fused = lstm_step_supported(B, H);
    for (int t = 0; t < T && fused; ++t) {
      const long o = static_cast<long>(t) * B;
      LAUNCH("lstm_step", t > 0 ? 8.0 * B * H * H : 0.0, (t > 0 ? 8.0 * H * H : 0.0) + 34.0 * B * H,
             lstm_step_fwd(zx + o * 4 * H, t > 0 ? hs + (o - B) * H : nullptr, static_cast<const bf16_t*>(wf(p + 1)),
                           t > 0 ? c + (o - B) * H : nullptr, B, H, gates + o * 4 * H, c + o * H, hs + o * H, ls_));
    }
    for (int t = 0; t < T && !fused; ++t) {
      float* zt = zx + static_cast<long>(t) * B * 4 * H;
      if (t > 0) {
        GemmDesc gh = gd(B, 4 * H, H, opK(hs + static_cast<long>(t - 1) * B * H, H), opK(wf(p + 1), H), 4 * H);
        gh.epi.res_f32 = zt;
        gh.epi.out_f32 = zt;
        gemm(gh);
      }
      LAUNCH("lstm_cell", 0, 0, lstm_cell_fwd(zt, t > 0 ? c + static_cast<long>(t - 1) * B * H : nullptr, B, H,
                              gates + static_cast<long>(t) * B * 4 * H, c + static_cast<long>(t) * B * H,
                              hs + static_cast<long>(t) * B * H, ls_));
    }
    LAUNCH("residual", 0, 6.0 * TB * H, add_bf16(static_cast<const bf16_t*>(u), hs, static_cast<bf16_t*>(out), TB * H, ls_));
    u = out;
  }
  if (ce) {
    GemmDesc gv = gd(static_cast<int>(TB), V, H, opK(u, H), opK(wf(3 * L), H), V);
    gv.epi.bias_bf16 = static_cast<const bf16_t*>(wf(3 * L + 1));
    gv.epi.out_f32 = ws<float>(1);
    gemm(gv);
    LAUNCH("softmax_ce", 0, ce_bytes(TB, V), softmax_ce(ws<float>(1), labels, static_cast<int>(TB), V, stash<void>(slot, 4 * L), 1, loss, ws<float>(7),
                         ls_));
  }
}

void Stage::bwd_lstm(int slot, const void* dy, void* dx) {
  const int L = d_.num_layers, B = d_.batch, I = d_.dims[0], H = d_.dims[1], T = d_.dims[2], V = d_.dims[3];
  const bool ce = d_.head == SPECTRAIN_HEAD_CE;
  const long TB = static_cast<long>(T) * B;
  const Slot& sl = slots_[slot];
  float* part = ws<float>(ws_colsum_);
  const void* du = dy;
  int pp = 2;
  if (ce) {
    const bf16_t* dl = stash<bf16_t>(slot, 4 * L);
    const void* uL = stash<void>(slot, 4 * (L - 1) + 3);
    GemmDesc gw = gd(V, H, static_cast<int>(TB), opR(dl, V), opR(uL, H), H);
    gw.epi.out_f32 = grad(3 * L);
    gemm(gw);
    LAUNCH("bias_grad", 0, colsum_bytes(TB, V, 2), column_sum(dl, 1, TB, V, V, grad(3 * L + 1), 0, part, s_));
    GemmDesc gx = gd(static_cast<int>(TB), H, V, opK(dl, V), opR(wb(3 * L), H), H);
    gx.epi.out_bf16 = ws<bf16_t>(pp);
    gemm(gx);
    du = ws<void>(pp);
    pp = 3;
  }
  bf16_t* dz = ws<bf16_t>(4);
  float* dh_rec = ws<float>(5);
  float* dc = ws<float>(6);
  for (int l = L - 1; l >= 0; --l) {
    const int p = 3 * l, q = 4 * l;
    const int in = l == 0 ? I : H;
    const void* u = l == 0 ? sl.x : stash<void>(slot, 4 * (l - 1) + 3);
    const float* gates = stash<float>(slot, q);
    const float* c = stash<float>(slot, q + 1);
    const bf16_t* hs = stash<bf16_t>(slot, q + 2);
    LAUNCH("clear_dc", 0, 4.0 * B * H, fill_f32(dc, 0.0f, static_cast<long>(B) * H, s_));
    const bool fused = lstm_step_supported(B, H);
    if (fused) {
      bf16_t* whT = ws<bf16_t>(8);
      LAUNCH("transpose", 0, 8.0 * H * H * 2, transpose_bf16(static_cast<const bf16_t*>(wb(p + 1)), 4 * H, H, whT, s_));
      for (int t = T - 1; t >= 0; --t) {
        const long o = static_cast<long>(t) * B;
        LAUNCH("lstm_step_bwd", t < T - 1 ? 8.0 * B * H * H : 0.0, (t < T - 1 ? 8.0 * H * H : 0.0) + 54.0 * B * H,
               lstm_step_bwd(t < T - 1 ? dz + (o + B) * 4 * H : nullptr, whT, static_cast<const bf16_t*>(du) + o * H,
                             gates + o * 4 * H, c + o * H, t > 0 ? c + (o - B) * H : nullptr, B, H, dc, dz + o * 4 * H,
                             s_));
      }
    }
    for (int t = T - 1; t >= 0 && !fused; --t) {
      const long o = static_cast<long>(t) * B;
      LAUNCH("lstm_cell_bwd", 0, 0, lstm_cell_bwd(static_cast<const bf16_t*>(du) + o * H, t < T - 1 ? dh_rec : nullptr, gates + o * 4 * H,
                              c + o * H, t > 0 ? c + (o - B) * H : nullptr, B, H, dc, dz + o * 4 * H, s_));
      if (t > 0) {
        GemmDesc gh = gd(B, H, 4 * H, opK(dz + o * 4 * H, 4 * H), opR(wb(p + 1), H), H);
        gh.epi.out_f32 = dh_rec;
        gemm(gh);
      }
    }
    GemmDesc wx = gd(4 * H, in, static_cast<int>(TB), opR(dz, 4 * H), opR(u, in), in);
    wx.epi.out_f32 = grad(p);
    gemm(wx);
    if (T > 1) {
      GemmDesc wh = gd(4 * H, H, static_cast<int>(TB - B), opR(dz + static_cast<long>(B) * 4 * H, 4 * H), opR(hs, H), H);
      wh.epi.out_f32 = grad(p + 1);
      gemm(wh);
    } else {
      LAUNCH("clear_grad", 0, 16.0 * H * H, fill_f32(grad(p + 1), 0.0f, 4L * H * H, s_));
    }
    LAUNCH("bias_grad", 0, colsum_bytes(TB, 4 * H, 2), column_sum(dz, 1, TB, 4 * H, 4 * H, grad(p + 2), 0, part, s_));
    if (l == 0 && !dx) break;
    void* out = l == 0 ? dx : ws<void>(pp);
    GemmDesc gxx = gd(static_cast<int>(TB), in, 4 * H, opK(dz, 4 * H), opR(wb(p), in), in);
    gxx.epi.res_bf16 = static_cast<const bf16_t*>(du);
    gxx.epi.out_bf16 = static_cast<bf16_t*>(out);
    gemm(gxx);
    du = out;
    pp = pp == 2 ? 3 : 2;
  }
}

}  // namespace spx
