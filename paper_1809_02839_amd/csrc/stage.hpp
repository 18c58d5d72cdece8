// One SpecTrain pipeline stage on one GPU: parameter arenas, activation
// stash ring and the per-kind forward/backward sequences of kernel launches.
#pragma once

#include <cstdint>
#include <cstdio>
#include <initializer_list>
#include <map>
#include <stdexcept>
#include <string>
#include <vector>

#include "../../include/spectrain.h"
#include "kernels.hpp"

#define LAUNCH(family, flops, bytes, expr) timed(family, flops, bytes, 0.0, [&]() { return (expr); })
// extra: bytes the launch moves beyond its algorithmic ones (reported apart)
#define LAUNCH_X(family, flops, bytes, extra, expr) timed(family, flops, bytes, extra, [&]() { return (expr); })

namespace spx {

// Failure carrying an ABI status code; caught at the C boundary.
struct StageError : std::runtime_error {
  int code;
  StageError(int c, const std::string& m) : std::runtime_error(m), code(c) {}
};

void hip_check(hipError_t e, const char* what);

// Bytes of the per-device scratch array of the allocation-free backward: the
// split-K workspace of a bf16 stage, so both backward entry points split
// every GEMM alike and give bitwise identical results.
constexpr size_t SCRATCH_BYTES = SPECTRAIN_NOALLOC_SCRATCH_BYTES;   // two halves: stage stream, side stream
// Device address of that array on `device` (looked up on first use, cached).
float* device_scratch(int device);

// A set of device sub-buffers carved from one hipMalloc, each 256-byte aligned.
class DeviceBlock {
 public:
  DeviceBlock() = default;
  DeviceBlock(const DeviceBlock&) = delete;
  DeviceBlock& operator=(const DeviceBlock&) = delete;
  DeviceBlock(DeviceBlock&& o) noexcept : base_(o.base_), total_(o.total_) { o.base_ = nullptr; o.total_ = 0; }
  size_t add(size_t bytes);  // returns an offset; call before allocate()
  void allocate();
  void release();
  template <typename T>
  T* at(size_t off) const { return reinterpret_cast<T*>(base_ + off); }
  size_t bytes() const { return total_; }
  ~DeviceBlock() { release(); }

 private:
  char* base_ = nullptr;
  size_t total_ = 0;
};

// Pinned, device-mapped host memory owned until destruction (also when the
// owning stage's constructor throws after allocating it).
class PinnedInts {
 public:
  PinnedInts() = default;
  PinnedInts(const PinnedInts&) = delete;
  PinnedInts& operator=(const PinnedInts&) = delete;
  void allocate(size_t n);   // zero-filled
  int* host() const { return host_; }
  int* dev() const { return dev_; }
  ~PinnedInts();

 private:
  int* host_ = nullptr;
  int* dev_ = nullptr;
};

struct TensorInfo {
  long off;   // element offset in the padded arenas
  long n;     // element count
};

class Stage {
 public:
  Stage(const spectrain_stage_desc& d, const float* W0, size_t n_params, hipStream_t s);
  ~Stage();

  size_t num_params() const { return n_params_; }
  void predict(int s, int slot);
  void forward(int64_t mb, const void* x, void* y, const int32_t* labels, float* loss);
  void backward(int64_t mb, const void* dy, void* dx);
  // The same backward with every split-K partial plane in the device's
  // scratch array instead of the stage's workspace; allocates nothing.
  void backward_noalloc(int64_t mb, const void* dy, void* dx);
  // The forward of mb_f and the backward of mb_b with the effect of forward()
  // then backward(): no update lies between the two in the stage's order, so
  // both read the weights of the same version, and they share no buffer. The
  // forward runs on a stream of its own with its own workspace copy, beside
  // the backward; the stage stream waits for both before the call's later
  // work.
  void forward_backward(int64_t mb_f, const void* x, void* y, const int32_t* labels, float* loss, int64_t mb_b,
                        const void* dy, void* dx);
  void update(int s_f, int s_b);
  void get_state(float* W, float* v);
  void set_state(const float* W, const float* v);
  void get_predicted(int slot, float* out);
  size_t read_stash(int64_t mb, int index, void* host, size_t capacity);
  bool nonfinite() const { return *reinterpret_cast<volatile int*>(flag_.host()) != 0; }
  void sync();
  // serial: every launch on the stage stream (forward_backward's forward and
  // the weight gradients included), for each launch's own duration
  void profile(bool enable, bool serial = false);
  int profile_read(spectrain_kernel_stat* out, int capacity);

 private:
  struct Slot {
    bool used = false;
    int64_t mb = -1;
    const void* x = nullptr;
    void* y = nullptr;
  };

  // ---- layout and buffers
  void build_layout();
  void plan_buffers();
  long tensor_off(int i) const { return tensors_[i].off; }
  const void* wf(int i) const;   // predicted slot 0 (forward) of tensor i
  const void* wb(int i) const;   // backward weights of tensor i (slot 1, or the mini-batch's stash)
  float* grad(int i) const { return g_ + tensors_[i].off; }
  template <typename T>
  T* stash(int slot, int buf) const { return slot_blocks_[slot].at<T>(stash_off_[buf]); }
  template <typename T>
  T* ws(int buf) const { return wsb_->at<T>(ws_off_[buf]); }
  // defer: the GEMM is the only writer of a gradient tensor (plain float32
  // store into g); when it splits K, its partials stay in the deferred buffer
  // and the update sums them instead of a separate reduction pass.
  void gemm(const GemmDesc& d, bool defer = false);
  // A weight-gradient GEMM on the side stream: it waits for everything issued
  // on the stage stream so far (its inputs) and runs beside the data-gradient
  // chain that follows; join_side() makes the stage stream wait for all of
  // the side stream's work (before a buffer those GEMMs read is rewritten,
  // and at the end of every backward).
  void side_gemm(const GemmDesc& d, std::initializer_list<const void*> reads);
  // Any launches issued by `issue` on the side stream (they launch on ls_).
  template <typename F>
  void on_side(std::initializer_list<const void*> reads, F&& issue) {
    if (serial_) {   // profiling one launch at a time: the side launches stay on the stage stream
      issue();
      return;
    }
    hip_check(hipEventRecord(fork_ev_, s_), "hipEventRecord");
    hip_check(hipStreamWaitEvent(s2_, fork_ev_, 0), "hipStreamWaitEvent");
    ls_ = s2_;
    try {
      issue();
    } catch (...) {
      ls_ = s_;
      throw;
    }
    ls_ = s_;
    side_pending_ = true;
    // completion event for the buffers read; a ring entry is recorded again
    // only after many later side launches, and a wait enqueued earlier
    // already refers to the record it saw
    hipEvent_t ev = side_ev_[side_next_];
    side_next_ = (side_next_ + 1) % side_ev_.size();
    hip_check(hipEventRecord(ev, s2_), "hipEventRecord");
    for (const void* b : reads) side_reads_[b] = ev;
  }
  void join_side();
  // The stage stream waits for the side-stream GEMMs that read `buf` before
  // it is rewritten (no-op when none is pending).
  void protect(const void* buf);

  // Launch wrapper: checks the launch status and, while profiling, brackets
  // the launch with events on the stage's stream.
  template <typename F>
  void timed(const char* family, double flops, double bytes, double extra, F&& launch) {
    if (!prof_on_) {
      hip_check(launch(), family);
      return;
    }
    hipEvent_t a = prof_event(), b = prof_event();
    hip_check(hipEventRecord(a, ls_), "hipEventRecord");
    hip_check(launch(), family);
    hip_check(hipEventRecord(b, ls_), "hipEventRecord");
    auto it = prof_index_.find(family);
    int fam;
    if (it == prof_index_.end()) {
      fam = static_cast<int>(prof_stats_.size());
      prof_index_[family] = fam;
      spectrain_kernel_stat k{};
      std::snprintf(k.name, sizeof(k.name), "%s", family);
      prof_stats_.push_back(k);
    } else {
      fam = it->second;
    }
    prof_recs_.push_back({fam, a, b, flops, bytes, extra});
  }
  hipEvent_t prof_event();
  void prof_collect();

  // ---- per kind
  void fwd_fc(int slot, const void* x, void* y, const int32_t* labels, float* loss);
  void bwd_fc(int slot, const void* dy, void* dx);
  void fwd_conv(int slot, const void* x, void* y, const int32_t* labels, float* loss);
  void bwd_conv(int slot, const void* dy, void* dx);
  void fwd_bneck(int slot, const void* x, void* y, const int32_t* labels, float* loss);
  void pool_head_fwd(int slot, const void* yl, int HW, int C, int t, int id_pool, int id_dl, int wsl,
                     const int32_t* labels, float* loss);
  void pool_head_bwd(int slot, const void* yl, int HW, int C, int t, int id_pool, int id_dl, int wsl, void* dz);
  void bwd_bneck(int slot, const void* dy, void* dx);
  void fwd_tfm(int slot, const void* x, void* y, const int32_t* labels, float* loss);
  void bwd_tfm(int slot, const void* dy, void* dx);
  void fwd_lstm(int slot, const void* x, void* y, const int32_t* labels, float* loss);
  void bwd_lstm(int slot, const void* dy, void* dx);

  spectrain_stage_desc d_;
  hipStream_t s_;
  int dt_;        // 1 = bf16 operands, 0 = float32
  size_t esz_;    // operand element size
  std::vector<TensorInfo> tensors_;
  size_t n_params_ = 0;
  long n_arena_ = 0;

  DeviceBlock arena_;
  float* W_ = nullptr;
  float* v_ = nullptr;
  float* g_ = nullptr;
  void* what_[2] = {nullptr, nullptr};
  DeviceBlock wstash_;                   // STASH policy: one weight copy per stash slot
  std::vector<size_t> wstash_off_;
  const void* bwd_weights_ = nullptr;    // base of the weights the current backward reads
  PinnedInts flag_;   // set by the update kernel on a non-finite value

  std::vector<Slot> slots_;
  std::vector<DeviceBlock> slot_blocks_;
  std::vector<size_t> stash_off_;
  std::vector<size_t> stash_bytes_;      // size of each stash buffer (0: unused for this stage)
  DeviceBlock ws_block_;
  std::vector<size_t> ws_off_;
  DeviceBlock ws_block_f_;               // workspace copy of a forward that runs beside a backward
  const DeviceBlock* wsb_ = &ws_block_;  // workspace of the pass being issued
  bool concurrent_ = false;              // issuing the passes of forward_backward (GEMM tile rule)
  // workspace ids after the kind's own buffers: column-sum partials of the
  // stage stream and of the side stream, split-K partials of each stream
  int ws_colsum_ = -1, ws_colsum2_ = -1, ws_split_ = -1, ws_split2_ = -1;
  size_t gemm_ws_bytes_ = 0;
  float* ext_ws_ = nullptr;              // split-K partials of the current call, when not the workspace
  hipStream_t s2_ = nullptr;             // side stream (weight gradients), default priority
  hipStream_t ls_ = nullptr;             // stream of the launch being issued: s_, s2_ or s3_
  hipStream_t s3_ = nullptr;             // forward beside a backward, default priority
  hipEvent_t ffork_ev_ = nullptr, fjoin_ev_ = nullptr;
  hipEvent_t fork_ev_ = nullptr, join_ev_ = nullptr;
  bool side_pending_ = false;
  std::vector<hipEvent_t> side_ev_;      // completion events of side GEMMs (a ring)
  size_t side_next_ = 0;
  std::map<const void*, hipEvent_t> side_reads_;   // buffer -> last side GEMM reading it
  int device_ = -1;                      // device current at create (the stream's device)
  bool g_pending_ = false;
  DeviceBlock defer_block_;              // split-K partials of gradients the update reduces
  float* defer_ = nullptr;
  long defer_cap_ = 0, defer_used_ = 0;  // floats
  std::vector<UpdateSegment> defer_segs_;

  struct ProfRec {
    int family;
    hipEvent_t a, b;
    double flops, bytes, extra;
  };
  bool prof_on_ = false;
  bool serial_ = false;                  // profile mode 2: every launch on the stage stream
  std::vector<hipEvent_t> prof_pool_;
  size_t prof_used_ = 0;
  std::vector<ProfRec> prof_recs_;
  std::vector<spectrain_kernel_stat> prof_stats_;
  std::map<std::string, int> prof_index_;
};

}  // namespace spx
