// Host runtime of the offloaded-MoE decode hot path: context, per-layer HBM
// slot pools, copy engine (pinned host -> device on a side stream, fenced by
// events), the layer orchestrator, event timing, and the C ABI of spp.h.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <chrono>
#include <immintrin.h>
#include <cmath>
#include <cstring>
#include <memory>
#include <new>
#include <string>
#include <vector>

#include "spp.h"
#include "spp_internal.h"
#include "spp_policy.h"

namespace {

thread_local std::string g_err;

spp_status fail(spp_status s, const std::string& m) {
  g_err = m;
  return s;
}

#define SPP_HIP(expr)                                                                              \
  do {                                                                                             \
    hipError_t e_ = (expr);                                                                        \
    if (e_ != hipSuccess) return fail(SPP_EHIP, std::string(#expr) + ": " + hipGetErrorString(e_)); \
  } while (0)

// Per layer call: start, routing result on the host, before/after the copy
// waits, FFN kernel begin/end (stamped by the kernel dispatch), end.
constexpr int kEvStart = 0, kEvRouted = 1, kEvWaitA = 2, kEvWaitB = 3, kEvFfnBegin = 4, kEvFfnEnd = 5, kEvEnd = 6,
              kEvLoaded = 7;  // after the on-demand loads enqueued on the compute stream, before the copy waits
constexpr int kNumEv = 8;

// Events recorded on the compute stream by default end with a system-scope
// release (an L2 writeback) that stalls the stream for 10-20 us after kernels
// that wrote a lot.  Events that only order copy-stream work after compute
// work (no data written before them is read by another agent through them)
// and timing events (read after the streams synchronised) skip it.  The
// per-slot copy events keep the default: the FFN reads the copied data.
constexpr unsigned kOrderEventFlags = hipEventDisableTiming | hipEventDisableSystemFence;
constexpr unsigned kTimingEventFlags = hipEventDisableSystemFence;

struct TimingSet {
  hipEvent_t ev[kNumEv] = {};
  int32_t l = -1;
  bool predicted = false;
  bool shared = false;  // on-demand copies enqueued while a prefetch copy was in flight on the link
  // batched steps with several on-demand rounds: (before, after) the copy
  // waits of rounds 1.. (inside the FFN span)
  std::vector<hipEvent_t> extra;
  int32_t extra_used = 0;
};

struct LayerState {
  bool bound = false;
  const void* router_w = nullptr;
  const void* A = nullptr;
  const void* Bm = nullptr;
  const void* proj = nullptr;
  const void* shared = nullptr;
  const uint8_t* host_store = nullptr;
  const uint8_t* host_store_dev = nullptr;  // its device-visible address (read by the copy kernel)
  uint8_t* slots = nullptr;
  std::unique_ptr<spp::SlotPolicy> policy;
  std::vector<hipEvent_t> slot_ready;  // recorded on the copy stream after a copy into the slot
  std::vector<hipEvent_t> slot_ready2; // the same on the second copy stream
  std::vector<int32_t> slot_event;     // the slot whose slot_ready covers this slot's last copy
  std::vector<char> slot_pending;      // that event may not have been waited on
  std::vector<char> slot_whole;        // last copy-stream copy: 0 two halves, 1 + s whole on copy stream s
  std::vector<char> slot_inline;       // loaded on the compute stream by this call (in order before its FFN)
  hipEvent_t last_read = nullptr;      // recorded on the compute stream after the layer's FFN
  bool last_read_valid = false;
  std::vector<int32_t> pending_prefetch;  // prefetched for this layer, not yet executed
  std::vector<int32_t> prev_T;            // routing of this layer at its last call [B*K]
  std::vector<float> prev_g;              // and its gates
};

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

}  // namespace

spp_status spp::set_error(spp_status s, const char* msg) { return fail(s, msg ? msg : ""); }

struct spp_ctx {
  spp_model_desc d{};
  int device = 0;
  int num_cu = 256;  // compute units of the device
  hipStream_t compute = nullptr;
  hipStream_t copy = nullptr;   // expert copies: first half of a blob, or the whole blob
  hipStream_t copy2 = nullptr;  // second half, so that one stream's per-copy gap overlaps the other's transfer
  size_t elem = 0, blob_bytes = 0, stride = 0;
  std::vector<LayerState> layers;
  float* u_dev = nullptr;      // [maxB, D] prologue output
  float* x_dev = nullptr;      // [maxB, D] router input
  float* zbuf = nullptr;       // [maxB, n + r]
  uint64_t* ztag = nullptr;    // [n + r] batch-1 router values tagged with their launch's seq (zero: none yet)
  uint8_t* res_dev = nullptr;  // topk [maxB*K] i32 | gates [maxB*K] f32 | s [n] f32
  size_t res_bytes = 0, off_gates = 0, off_s = 0;
  // host records written by the router kernels (pinned, host-mapped):
  // routing [maxB*K][2] then priorities [n], each (seq << 32) | payload
  uint64_t* rec_host = nullptr;
  uint64_t* rec_host_dev = nullptr;  // device-visible address of rec_host
  size_t rec_count = 0;
  std::vector<int32_t> host_T;  // the last routing read from the records [maxB*K]
  std::vector<float> host_g;    // its gates
  std::vector<float> host_s;    // the last priorities [n]
  uint32_t router_seq = 0;  // last sequence number handed to a router launch
  int32_t prefetch_source = SPP_PREFETCH_ADAPTER;
  int32_t copy_engine = SPP_COPY_SPLIT;
  hipEvent_t demand_done = nullptr;  // on the compute stream after the latest on-demand copy kernels
  bool demand_done_valid = false;
  // batch-1 FFN split (spp_set_ffn_overlap): the experts already resident run on
  // compute2 while the on-demand copies run on the compute stream
  bool ffn_overlap = false;
  bool prefetch_parallel = false;  // whole prefetches of one call alternate the copy streams
  hipStream_t compute2 = nullptr;
  hipEvent_t route_done = nullptr;  // compute stream, after the router launch
  hipEvent_t hits_done = nullptr;   // compute2, after the resident experts' FFN launch
  unsigned* counter = nullptr;
  std::chrono::steady_clock::time_point t_grouped_launched{};  // the first grouped FFN launch's return
  float* partial = nullptr;    // [ffn_max_grid, D]
  uint8_t* probe_dev = nullptr;  // one blob, for copy profiling
  // batched decode (B > 1, bf16): expert groups and partial outputs
  bool grouped = false;
  int max_groups = 0, max_nsplit = 0;
  spp::GroupDesc* groups_dev = nullptr;   // device address of groups_host (host-mapped)
  spp::GroupDesc* groups_host = nullptr;  // per-layer group list, pinned and device-mapped: the grouped
                                          // kernel reads it in place (rewritten only after the next
                                          // router, i.e. after the previous FFN, has finished)
  float* ypart = nullptr;
  std::vector<hipEvent_t> round_done;  // per on-demand round: its FFN launch finished
  std::vector<int32_t> grp_start, grp_fill, grp_order;  // group building scratch (per call)
  std::vector<int> grp_rstart, grp_rcount;
  int64_t clock = 0;
  int ffn_wgs = 512;  // about this many workgroups share one batch-1 FFN launch (bf16/fp32 experts)
  // test hooks
  bool poison = false;
  int32_t copy_delay_us = 0;
  bool tier_serial = false;  // storage emulation: every expert read through the copy streams' one queue
  uint64_t wall_khz = 0;
  // last call record
  std::vector<spp::Transfer> last_loads, last_pref;
  std::vector<float> last_s;
  int32_t last_B = 0;
  bool logits_valid = false;  // zbuf still holds the last call's router logits
  bool last_s_valid = false;
  // timing
  bool timing = false;
  int32_t timing_level = 0;
  hipEvent_t pf_done[2] = {nullptr, nullptr};  // copy streams, after the latest prefetch copies (timing only)
  bool pf_done_valid = false;
  // per-layer totals of the timed calls (spp_get_layer_times)
  std::vector<int64_t> lt_calls, lt_latency_calls;
  std::vector<double> lt_exposed, lt_latency;
  std::vector<int32_t> pred_top;  // Top_{K+2}(s) of the last prediction (timing only), for layer pred_target
  int32_t pred_target = -1;
  std::vector<TimingSet> pending_sets, free_sets;
  bool have_prev = false;
  TimingSet prev{};
  spp_run_stats stats{};
};

namespace {

// Batched contexts (bf16, max_batch > 1, D % 256 == 0, I % 16 == 0) store
// experts in the tiled layout the grouped MFMA kernel streams linearly.
bool tiled_layout(const spp_model_desc& d) {
  return d.expert_codec == SPP_CODEC_PLAIN && d.max_batch > 1 && d.dtype == SPP_DTYPE_BF16 && d.D % 256 == 0 &&
         d.I % 16 == 0;
}

// Bytes of one expert blob (before the 4 KiB stride rounding).
size_t expert_bytes(const spp_model_desc& d) {
  if (d.expert_codec == SPP_CODEC_Q4)
    return static_cast<size_t>(d.I) * (3 * static_cast<size_t>(d.D) / 2 + 3 * static_cast<size_t>(d.D / 32) * 2);
  return static_cast<size_t>(3) * d.I * d.D * (d.dtype == SPP_DTYPE_BF16 ? 2 : 4);
}

bool desc_ok(const spp_model_desc* d, std::string* why) {
  if (!d) return *why = "desc is NULL", false;
  if (d->dtype != SPP_DTYPE_F32 && d->dtype != SPP_DTYPE_BF16) return *why = "dtype must be 0 (f32) or 1 (bf16)", false;
  const int elem = d->dtype == SPP_DTYPE_BF16 ? 2 : 4;
  if (d->L < 1 || d->D < 1 || d->n < 1 || d->K < 1 || d->I < 1 || d->S < 1 || d->max_batch < 1)
    return *why = "L, D, n, K, I, S, max_batch must be >= 1", false;
  if ((static_cast<int64_t>(d->D) * elem) % 16 != 0) return *why = "D * element size must be a multiple of 16 bytes", false;
  const int nch = (d->D * elem / 16 + 63) / 64;
  if (nch > 8) return *why = "D too large (at most 4096 bf16 / 2048 fp32)", false;
  if (d->max_batch > 1 && d->D % 16 != 0) return *why = "max_batch > 1 needs D a multiple of 16", false;
  if (d->n > spp::kMaxExpertsTopK) return *why = "n must be <= 1024", false;
  if (d->K > d->n || d->K > 32) return *why = "K must be <= min(n, 32)", false;
  if (d->r < 0 || d->r > 256) return *why = "r must be in [0, 256]", false;
  if ((static_cast<int64_t>(d->n) * d->r * elem) % 16 != 0) return *why = "n * r * element size must be a multiple of 16 bytes", false;
  if (d->n_shared < 0 || d->K + d->n_shared > spp::kMaxWork) return *why = "K + n_shared must be <= 32", false;
  if (d->has_proj != 0 && d->has_proj != 1) return *why = "has_proj must be 0 or 1", false;
  if (!(d->rms_eps >= 0.f) || !std::isfinite(d->rms_eps)) return *why = "rms_eps must be finite and >= 0", false;
  if (d->expert_codec != SPP_CODEC_PLAIN && d->expert_codec != SPP_CODEC_Q4)
    return *why = "expert_codec must be SPP_CODEC_PLAIN or SPP_CODEC_Q4", false;
  if (d->expert_codec == SPP_CODEC_Q4 && (d->dtype != SPP_DTYPE_BF16 || d->max_batch != 1 || d->D % 256 != 0))
    return *why = "4-bit experts need dtype bf16, max_batch 1 and D a multiple of 256", false;
  // only the tiled batched path runs a step in rounds; elsewhere every distinct
  // routed expert of a call must fit in the slots at once
  if (!tiled_layout(*d) && static_cast<int64_t>(d->S) < std::min<int64_t>(d->n, static_cast<int64_t>(d->K) * d->max_batch))
    return *why = "S must be >= min(n, K * max_batch) unless the experts use the tiled batched layout", false;
  return true;
}

spp_status check_ctx(spp_ctx* c) {
  if (!c) return fail(SPP_EINVAL, "ctx is NULL");
  return SPP_OK;
}

spp_status check_layer(spp_ctx* c, int32_t l, bool need_bound) {
  if (!c) return fail(SPP_EINVAL, "ctx is NULL");
  if (l < 0 || l >= c->d.L) return fail(SPP_EINVAL, "layer index out of range");
  if (need_bound && !c->layers[l].bound) return fail(SPP_ESTATE, "layer not bound");
  return SPP_OK;
}

spp_status take_set(spp_ctx* c, TimingSet* out) {
  if (!c->free_sets.empty()) {
    *out = c->free_sets.back();
    c->free_sets.pop_back();
    out->extra_used = 0;
    return SPP_OK;
  }
  TimingSet s;
  for (int i = 0; i < kNumEv; ++i) SPP_HIP(hipEventCreateWithFlags(&s.ev[i], kTimingEventFlags));
  *out = s;
  return SPP_OK;
}

float elapsed(hipEvent_t a, hipEvent_t b) {
  float ms = 0.f;
  if (hipEventElapsedTime(&ms, a, b) != hipSuccess) return 0.f;
  return ms;
}

// Fold the first `count` pending sets (all complete) into the totals.
void harvest(spp_ctx* c, size_t count) {
  for (size_t i = 0; i < count; ++i) {
    TimingSet& s = c->pending_sets[i];
    spp_run_stats& st = c->stats;
    st.router_us += 1e3 * elapsed(s.ev[kEvStart], s.ev[kEvRouted]);
    const double exposed = 1e3 * elapsed(s.ev[kEvWaitA], s.ev[kEvWaitB]);
    const double loads = 1e3 * elapsed(s.ev[kEvWaitA], s.ev[kEvLoaded]);
    double extra = 0.0;
    for (int32_t q = 0; q + 1 < s.extra_used; q += 2) extra += 1e3 * elapsed(s.extra[q], s.extra[q + 1]);
    st.exposed_us += exposed + extra;
    if (s.shared) {
      st.exposed_shared_us += loads + extra;
      st.shared_calls += 1;
    } else {
      st.exposed_load_us += loads + extra;
    }
    st.exposed_wait_us += exposed - loads;
    c->lt_calls[s.l] += 1;
    c->lt_exposed[s.l] += exposed + extra;
    st.ffn_us += 1e3 * elapsed(s.ev[kEvFfnBegin], s.ev[kEvFfnEnd]) - extra;
    st.tail_us += 1e3 * elapsed(s.ev[kEvFfnEnd], s.ev[kEvEnd]);
    if (c->have_prev) {
      const double span = 1e3 * elapsed(c->prev.ev[kEvStart], s.ev[kEvStart]);
      st.span_us += span;
      c->lt_latency[c->prev.l] += span;
      c->lt_latency_calls[c->prev.l] += 1;
      if (c->prev.predicted && s.l == c->prev.l + 1) {
        // W_l = t_exec(l+1) - t_pred(l); the compute window excludes the copy stalls inside it
        const double w = 1e3 * elapsed(c->prev.ev[kEvRouted], s.ev[kEvFfnBegin]);
        const double prev_exposed = 1e3 * elapsed(c->prev.ev[kEvWaitA], c->prev.ev[kEvWaitB]);
        st.window_us += w;
        st.compute_window_us += w - prev_exposed - exposed;
        st.window_samples += 1;
      }
      c->free_sets.push_back(c->prev);
    }
    c->prev = s;
    c->have_prev = true;
  }
  c->pending_sets.erase(c->pending_sets.begin(), c->pending_sets.begin() + count);
}

// One contiguous part of an expert blob from the offload tier (host offset
// `src_off`) into device memory, on a copy stream.  The copy kernel moves
// whole 16-byte chunks: a part is rounded up to 16 bytes, which stays inside
// the blob stride on both sides (the stride is a multiple of 4 KiB).
constexpr int kCopyWgs = 32;        // per half blob on a copy stream
constexpr int kInlineCopyWgs = 64;  // on-demand loads on the compute stream
hipError_t copy_part(spp_ctx* c, const LayerState& ls, uint8_t* dst, size_t src_off, size_t bytes, hipStream_t st) {
  if (c->copy_engine != SPP_COPY_KERNEL)
    return hipMemcpyAsync(dst, ls.host_store + src_off, bytes, hipMemcpyHostToDevice, st);
  spp::CopyList one{};
  one.src[0] = ls.host_store_dev + src_off;
  one.dst[0] = dst;
  one.n = 1;
  one.n16 = round_up(bytes, 16) / 16;
  return spp::launch_h2d_copies(one, kCopyWgs, st);
}

// Enqueue the copies `xs` into layer `ls`'s slots on the copy streams (a blob
// in two halves, one per stream, or whole on the first stream), after `war`
// (the last kernel that read this layer's slots).  demand: on-demand loads, which the compute
// stream waits for as a group, so one event after the last copy covers them
// (the streams are in order); otherwise prefetches, consumed one by one, each
// with its own event.  An event wait costs the host ~14 us while the event is
// pending, ~0.2 us once it completed, so every wait is preceded by a query.
spp_status copy_streams_wait(spp_ctx* c, hipEvent_t e) {
  if (e && hipEventQuery(e) != hipSuccess) {
    SPP_HIP(hipStreamWaitEvent(c->copy, e, 0));
    SPP_HIP(hipStreamWaitEvent(c->copy2, e, 0));
  }
  return SPP_OK;
}

spp_status issue_copies(spp_ctx* c, LayerState& ls, const std::vector<spp::Transfer>& xs, hipEvent_t war,
                        bool demand) {
  if (xs.empty()) return SPP_OK;
  // WAR on slot reuse, unless the last kernel that read this layer already finished
  if (spp_status e = copy_streams_wait(c, war)) return e;
  // prefetches start once the on-demand loads on the compute stream are done:
  // both cross the same host link, and the on-demand loads are the ones the
  // next kernel waits for
  if (!demand && c->demand_done_valid)
    if (spp_status e = copy_streams_wait(c, c->demand_done)) return e;
  const int32_t last = xs.back().slot;
  // Copies go out as two halves of every blob, one per copy stream (the split
  // is 4 KiB aligned), so that one stream's per-copy gap overlaps the other's
  // transfer -- except prefetches beside copy-kernel loads, which go out whole
  // and in issue order on the first copy stream.  Serial prefetches finish
  // the one needed first (this layer's before the next layer's) at the link's
  // full rate instead of sharing it; that and one DMA fixed cost per expert
  // instead of two gave +3-4% tokens/s at M_max 1 on the recall-calibrated
  // 4-bit workloads against halves or whole copies alternating the streams.
  const bool whole = !demand && c->copy_engine == SPP_COPY_SPLIT && !c->tier_serial;
  const size_t half = whole ? c->blob_bytes : (c->blob_bytes / 2 + 4095) / 4096 * 4096;
  const size_t part[2] = {std::min(half, c->blob_bytes), c->blob_bytes - std::min(half, c->blob_bytes)};
  const hipStream_t cs[2] = {c->copy, c->copy2};
  int k_whole = 0;
  for (const spp::Transfer& t : xs) {
    uint8_t* dst = ls.slots + static_cast<size_t>(t.slot) * c->stride;
    // a whole copy goes to stream ws (the second one for every other copy of
    // this call with spp_set_prefetch_parallel); halves: stream h carries part h
    const int ws = whole && c->prefetch_parallel ? (k_whole & 1) : 0;
    const char code = whole ? static_cast<char>(1 + ws) : 0;
    const hipStream_t streams[2] = {whole ? cs[ws] : c->copy, c->copy2};
    if (ls.slot_pending[t.slot] && ls.slot_whole[t.slot] != code) {
      // WAW after a change of stream assignment (copy engine, storage
      // emulation, parallel prefetches): an earlier copy into this slot that
      // was never waited on may still be in flight on a stream that the new
      // copy's streams are not ordered behind.  Each stream of the new copy
      // waits for the old copy's events recorded on the other stream.
      const int32_t ev = ls.slot_event[t.slot];
      const char old = ls.slot_whole[t.slot];
      for (int os = 0; os < 2; ++os) {
        const bool old_on = old == 0 || old == 1 + os;
        if (!old_on) continue;
        const hipEvent_t e = old == 0 && os == 1 ? ls.slot_ready2[ev] : ls.slot_ready[ev];
        for (int ns = 0; ns < 2; ++ns) {
          const bool new_on = code == 0 || code == 1 + ns;
          if (new_on && ns != os && hipEventQuery(e) != hipSuccess) SPP_HIP(hipStreamWaitEvent(cs[ns], e, 0));
        }
      }
    }
    for (int h = 0; h < 2; ++h) {
      if (part[h] == 0) continue;
      if (c->copy_delay_us > 0) {
        const uint64_t ticks = c->wall_khz * static_cast<uint64_t>(c->copy_delay_us) / 1000;
        SPP_HIP(spp::launch_spin(ticks, static_cast<uint32_t>(c->copy_delay_us) * 64u + 1024u, streams[h]));
      }
      const size_t off = h == 0 ? 0 : part[0];
      if (c->poison) SPP_HIP(hipMemsetAsync(dst + off, 0xFF, part[h], streams[h]));
      SPP_HIP(copy_part(c, ls, dst + off, static_cast<size_t>(t.expert) * c->stride + off, part[h], streams[h]));
    }
    if (!demand || t.slot == last) {
      // a whole copy has one event, slot_ready on its stream; readers skip
      // slot_ready2 (a wait on a pending event costs ~12 us of host time)
      SPP_HIP(hipEventRecord(ls.slot_ready[t.slot], streams[0]));
      if (!whole) SPP_HIP(hipEventRecord(ls.slot_ready2[t.slot], c->copy2));
    }
    if (whole) ++k_whole;
    ls.slot_event[t.slot] = demand ? last : t.slot;
    ls.slot_pending[t.slot] = 1;
    ls.slot_whole[t.slot] = code;
    c->stats.copies += 1;
    c->stats.copy_bytes += static_cast<int64_t>(c->blob_bytes);
  }
  return SPP_OK;
}

// On-demand loads on the compute stream (SPP_COPY_SPLIT): copy-list kernels
// ahead of the FFN that reads the slots, which the stream order then fences
// (RAW) as it fences their overwrite after the previous FFN (WAR).  A slot
// whose earlier copy on the copy streams may still be in flight is waited for
// first (WAW).
spp_status issue_inline(spp_ctx* c, LayerState& ls, const std::vector<spp::Transfer>& xs) {
  if (xs.empty()) return SPP_OK;
  std::vector<int32_t> waited;
  for (const spp::Transfer& t : xs) {
    if (!ls.slot_pending[t.slot]) continue;
    const int32_t ev = ls.slot_event[t.slot];
    if (std::find(waited.begin(), waited.end(), ev) == waited.end()) {
      if (hipEventQuery(ls.slot_ready[ev]) != hipSuccess) SPP_HIP(hipStreamWaitEvent(c->compute, ls.slot_ready[ev], 0));
      if ((!ls.slot_whole[ev] && hipEventQuery(ls.slot_ready2[ev]) != hipSuccess))
        SPP_HIP(hipStreamWaitEvent(c->compute, ls.slot_ready2[ev], 0));
      waited.push_back(ev);
    }
    ls.slot_pending[t.slot] = 0;
  }
  spp::CopyList list{};
  list.n16 = round_up(c->blob_bytes, 16) / 16;
  for (size_t i = 0; i < xs.size(); ++i) {
    const spp::Transfer& t = xs[i];
    uint8_t* dst = ls.slots + static_cast<size_t>(t.slot) * c->stride;
    if (c->copy_delay_us > 0) {
      const uint64_t ticks = c->wall_khz * static_cast<uint64_t>(c->copy_delay_us) / 1000;
      SPP_HIP(spp::launch_spin(ticks, static_cast<uint32_t>(c->copy_delay_us) * 64u + 1024u, c->compute));
    }
    if (c->poison) SPP_HIP(hipMemsetAsync(dst, 0xFF, c->blob_bytes, c->compute));
    list.src[list.n] = ls.host_store_dev + static_cast<size_t>(t.expert) * c->stride;
    list.dst[list.n] = dst;
    ++list.n;
    // a delayed copy goes out alone, right after its delay
    if (list.n == spp::kMaxCopyList || i + 1 == xs.size() || c->copy_delay_us > 0) {
      SPP_HIP(spp::launch_h2d_copies(list, kInlineCopyWgs, c->compute));
      list.n = 0;
    }
    ls.slot_inline[t.slot] = 1;
    c->stats.copies += 1;
    c->stats.copy_bytes += static_cast<int64_t>(c->blob_bytes);
  }
  SPP_HIP(hipEventRecord(c->demand_done, c->compute));
  c->demand_done_valid = true;
  return SPP_OK;
}

// The on-demand loads of one round: on the compute stream (SPP_COPY_SPLIT) or
// on the copy streams after `war`.
spp_status issue_demand(spp_ctx* c, LayerState& ls, const std::vector<spp::Transfer>& xs, hipEvent_t war) {
  if (c->copy_engine == SPP_COPY_SPLIT && !c->tier_serial) return issue_inline(c, ls, xs);
  return issue_copies(c, ls, xs, war, true);
}

spp_status sync_all(spp_ctx* c) {
  SPP_HIP(hipStreamSynchronize(c->copy));
  SPP_HIP(hipStreamSynchronize(c->copy2));
  SPP_HIP(hipStreamSynchronize(c->compute2));
  SPP_HIP(hipStreamSynchronize(c->compute));
  return SPP_OK;
}


// Synchronous fill of slots from the host store according to the policy table.
spp_status fill_slots(spp_ctx* c, LayerState& ls, const std::vector<int32_t>& before) {
  const auto& table = ls.policy->slot_experts();
  for (int32_t j = 0; j < c->d.S; ++j) {
    ls.slot_pending[j] = 0;
    ls.slot_inline[j] = 0;
    if (table[j] == spp::kEmpty || table[j] == before[j]) continue;
    SPP_HIP(hipMemcpy(ls.slots + static_cast<size_t>(j) * c->stride,
                      ls.host_store + static_cast<size_t>(table[j]) * c->stride, c->blob_bytes,
                      hipMemcpyHostToDevice));
  }
  return SPP_OK;
}

void free_ctx(spp_ctx* c) {
  if (!c) return;
  if (c->copy) (void)hipStreamSynchronize(c->copy);
  if (c->copy2) (void)hipStreamSynchronize(c->copy2);
  if (c->compute2) (void)hipStreamSynchronize(c->compute2);
  (void)hipStreamSynchronize(c->compute);
  for (LayerState& ls : c->layers) {
    if (ls.slots) (void)hipFree(ls.slots);
    for (hipEvent_t e : ls.slot_ready)
      if (e) (void)hipEventDestroy(e);
    for (hipEvent_t e : ls.slot_ready2)
      if (e) (void)hipEventDestroy(e);
    if (ls.last_read) (void)hipEventDestroy(ls.last_read);
  }
  auto destroy_set = [](TimingSet& s) {
    for (hipEvent_t e : s.ev)
      if (e) (void)hipEventDestroy(e);
    for (hipEvent_t e : s.extra)
      if (e) (void)hipEventDestroy(e);
  };
  for (auto* v : {&c->pending_sets, &c->free_sets})
    for (TimingSet& s : *v) destroy_set(s);
  if (c->have_prev) destroy_set(c->prev);
  for (hipEvent_t e : c->round_done)
    if (e) (void)hipEventDestroy(e);
  if (c->demand_done) (void)hipEventDestroy(c->demand_done);
  if (c->route_done) (void)hipEventDestroy(c->route_done);
  if (c->hits_done) (void)hipEventDestroy(c->hits_done);
  for (hipEvent_t e : c->pf_done)
    if (e) (void)hipEventDestroy(e);
  for (void* p : {static_cast<void*>(c->u_dev), static_cast<void*>(c->x_dev), static_cast<void*>(c->zbuf),
                  static_cast<void*>(c->ztag), static_cast<void*>(c->res_dev), static_cast<void*>(c->counter),
                  static_cast<void*>(c->partial), static_cast<void*>(c->probe_dev)})
    if (p) (void)hipFree(p);
  if (c->rec_host) (void)hipHostFree(c->rec_host);
  if (c->groups_host) (void)hipHostFree(c->groups_host);
  if (c->ypart) (void)hipFree(c->ypart);
  if (c->copy) (void)hipStreamDestroy(c->copy);
  if (c->copy2) (void)hipStreamDestroy(c->copy2);
  if (c->compute2) (void)hipStreamDestroy(c->compute2);
  delete c;
}

spp_status create_impl(const spp_model_desc* desc, void* stream, spp_ctx** out) {
  std::string why;
  if (!out) return fail(SPP_EINVAL, "out is NULL");
  *out = nullptr;
  if (!desc_ok(desc, &why)) return fail(SPP_EINVAL, why);
  std::unique_ptr<spp_ctx, void (*)(spp_ctx*)> c(new (std::nothrow) spp_ctx(), free_ctx);
  if (!c) return fail(SPP_ENOMEM, "host allocation failed");
  c->d = *desc;
  SPP_HIP(hipGetDevice(&c->device));
  SPP_HIP(hipDeviceGetAttribute(&c->num_cu, hipDeviceAttributeMultiprocessorCount, c->device));
  c->compute = static_cast<hipStream_t>(stream);
  c->elem = desc->dtype == SPP_DTYPE_BF16 ? 2 : 4;
  c->blob_bytes = expert_bytes(*desc);
  c->stride = round_up(c->blob_bytes, 4096);
  SPP_HIP(hipStreamCreateWithFlags(&c->copy, hipStreamNonBlocking));
  SPP_HIP(hipStreamCreateWithFlags(&c->copy2, hipStreamNonBlocking));
  SPP_HIP(hipEventCreateWithFlags(&c->demand_done, kOrderEventFlags));
  SPP_HIP(hipStreamCreateWithFlags(&c->compute2, hipStreamNonBlocking));
  SPP_HIP(hipEventCreateWithFlags(&c->route_done, kOrderEventFlags));
  SPP_HIP(hipEventCreateWithFlags(&c->hits_done, kOrderEventFlags));
  for (hipEvent_t& e : c->pf_done) SPP_HIP(hipEventCreateWithFlags(&e, kOrderEventFlags));
  const spp_model_desc& d = c->d;
  c->layers.resize(d.L);
  c->lt_calls.assign(d.L, 0);
  c->lt_latency_calls.assign(d.L, 0);
  c->lt_exposed.assign(d.L, 0.0);
  c->lt_latency.assign(d.L, 0.0);
  for (LayerState& ls : c->layers) {
    ls.policy.reset(new spp::SlotPolicy(d.S, d.n));
    if (hipMalloc(&ls.slots, c->stride * d.S) != hipSuccess) return fail(SPP_ENOMEM, "slot pool allocation failed");
    ls.slot_ready.assign(d.S, nullptr);
    ls.slot_ready2.assign(d.S, nullptr);
    ls.slot_pending.assign(d.S, 0);
    ls.slot_whole.assign(d.S, 0);
    ls.slot_inline.assign(d.S, 0);
    ls.slot_event.resize(d.S);
    for (int32_t j = 0; j < d.S; ++j) ls.slot_event[j] = j;
    for (hipEvent_t& e : ls.slot_ready) SPP_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));
    for (hipEvent_t& e : ls.slot_ready2) SPP_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));
    SPP_HIP(hipEventCreateWithFlags(&ls.last_read, kOrderEventFlags));
  }
  const size_t BD = static_cast<size_t>(d.max_batch) * d.D;
  if (hipMalloc(&c->u_dev, BD * sizeof(float)) != hipSuccess ||
      hipMalloc(&c->x_dev, BD * sizeof(float)) != hipSuccess ||
      hipMalloc(&c->zbuf, static_cast<size_t>(d.max_batch) * (d.n + d.r) * sizeof(float)) != hipSuccess ||
      hipMalloc(&c->ztag, static_cast<size_t>(d.n + d.r) * sizeof(uint64_t)) != hipSuccess ||
      hipMalloc(&c->partial, spp::ffn_max_grid() * d.D * sizeof(float)) != hipSuccess ||
      hipMalloc(&c->counter, 256) != hipSuccess)
    return fail(SPP_ENOMEM, "scratch allocation failed");
  const size_t bk = static_cast<size_t>(d.max_batch) * d.K;
  c->off_gates = round_up(bk * sizeof(int32_t), 64);
  c->off_s = c->off_gates + round_up(bk * sizeof(float), 64);
  c->res_bytes = c->off_s + round_up(static_cast<size_t>(d.n) * sizeof(float), 64);
  if (hipMalloc(&c->res_dev, c->res_bytes) != hipSuccess) return fail(SPP_ENOMEM, "result buffer allocation failed");
  c->rec_count = 2 * bk + static_cast<size_t>(d.n);
  if (hipHostMalloc(&c->rec_host, c->rec_count * sizeof(uint64_t), hipHostMallocMapped | hipHostMallocCoherent) !=
      hipSuccess)
    return fail(SPP_ENOMEM, "pinned record buffer allocation failed");
  SPP_HIP(hipHostGetDevicePointer(reinterpret_cast<void**>(&c->rec_host_dev), c->rec_host, 0));
  std::memset(c->rec_host, 0, c->rec_count * sizeof(uint64_t));  // sequence 0 is never handed out
  c->host_T.assign(bk, 0);
  c->host_g.assign(bk, 0.f);
  c->host_s.assign(d.n, 0.f);
  // batched decode runs the routed experts as grouped MFMA contractions
  c->grouped = tiled_layout(d);
  if (c->grouped) {
    c->max_groups = d.max_batch * d.K + d.n_shared * ((d.max_batch + spp::kGroupTokens - 1) / spp::kGroupTokens);
    c->max_nsplit = (d.I + 63) / 64;
    const size_t npairs = static_cast<size_t>(d.max_batch) * (d.K + d.n_shared);
    if (hipHostMalloc(&c->groups_host, sizeof(spp::GroupDesc) * c->max_groups,
                      hipHostMallocMapped | hipHostMallocCoherent) != hipSuccess ||
        hipMalloc(&c->ypart, npairs * c->max_nsplit * d.D * sizeof(float)) != hipSuccess)
      return fail(SPP_ENOMEM, "batched-decode buffers allocation failed");
    SPP_HIP(hipHostGetDevicePointer(reinterpret_cast<void**>(&c->groups_dev), c->groups_host, 0));
  }
  SPP_HIP(hipMemset(c->counter, 0, 256));
  SPP_HIP(hipMemset(c->ztag, 0, static_cast<size_t>(d.n + d.r) * sizeof(uint64_t)));  // seq 0 is never handed out
  SPP_HIP(hipMemset(c->res_dev, 0, c->res_bytes));
  c->last_s.assign(d.n, 0.f);
  SPP_HIP(hipDeviceSynchronize());
  *out = c.release();
  return SPP_OK;
}

// Hand the next sequence number to a router launch (never 0, the initial flag).
uint32_t next_router_seq(spp_ctx* c) {
  if (++c->router_seq == 0) c->router_seq = 1;
  return c->router_seq;
}

// Wait until the router launch tagged `seq` has written its host records:
// kind 0 the routing of B tokens (expert and gate of every (b, k)), kind 1 the
// priorities s; then copy their payloads into host_T / host_g or host_s.  A
// record is this launch's once its high half equals seq; records only ever
// move on to a newer launch's, so the scan resumes where it stopped.  After
// about 20 ms of spinning (queued work ahead of the router) the wait blocks on
// the stream instead; records still missing then are an error.
spp_status wait_router(spp_ctx* c, uint32_t seq, int kind, int32_t B) {
  // record arrays: expert ids [max_batch*K], gates [max_batch*K], priorities [n]
  const size_t bkmax = static_cast<size_t>(c->d.max_batch) * c->d.K;
  const size_t bk = static_cast<size_t>(B) * c->d.K;
  const uint64_t* const part[2] = {kind == 0 ? c->rec_host : c->rec_host + 2 * bkmax,
                                   kind == 0 ? c->rec_host + bkmax : nullptr};
  const size_t count = kind == 0 ? bk : static_cast<size_t>(c->d.n);
  const auto t0 = std::chrono::steady_clock::now();
  for (int q = 0; q < 2 && part[q]; ++q) {
    const uint64_t* rec = part[q];
    size_t i = 0;
    for (uint32_t it = 1; i < count; ++it) {
      if (static_cast<uint32_t>(__atomic_load_n(rec + i, __ATOMIC_ACQUIRE) >> 32) == seq) {
        ++i;
        continue;
      }
      if ((it & 1023u) == 0 && std::chrono::steady_clock::now() - t0 > std::chrono::milliseconds(20)) break;
      _mm_pause();
    }
    if (i < count) {
      SPP_HIP(hipStreamSynchronize(c->compute));
      for (; i < count; ++i)
        if (static_cast<uint32_t>(__atomic_load_n(rec + i, __ATOMIC_ACQUIRE) >> 32) != seq)
          return fail(SPP_EHIP, "router results were not written by the router launch");
    }
  }
  if (kind == 0) {
    for (size_t j = 0; j < bk; ++j) {
      c->host_T[j] = static_cast<int32_t>(static_cast<uint32_t>(part[0][j]));
      const uint32_t gb = static_cast<uint32_t>(part[1][j]);
      std::memcpy(&c->host_g[j], &gb, sizeof(float));
    }
  } else {
    for (size_t j = 0; j < count; ++j) {
      const uint32_t sb = static_cast<uint32_t>(part[0][j]);
      std::memcpy(&c->host_s[j], &sb, sizeof(float));
    }
  }
  return SPP_OK;
}

// Whether a prefetch copy enqueued by an earlier layer call may still be
// moving data over the host link (timing only: the events exist then).
bool prefetch_in_flight(spp_ctx* c) {
  if (!c->pf_done_valid) return false;
  return hipEventQuery(c->pf_done[0]) != hipSuccess || hipEventQuery(c->pf_done[1]) != hipSuccess;
}

// RAW: the compute stream waits for the copies into the slots a round reads.
// Every slot of the round leaves it no longer pending: the compute stream is
// then ordered behind its copy, by the stream order (loaded on it), by a wait
// enqueued here, or because the copy had already completed.  A slot left
// pending after its group's event was waited on would later query that
// event again after a new copy into the event's own slot re-recorded it, and
// wait for that unrelated copy.
spp_status wait_round(spp_ctx* c, LayerState& ls, const spp::Round& round, spp_layer_stats* st) {
  std::vector<int32_t> waited;  // each covering event is waited on once
  for (const auto& es : round) {
    const int32_t slot = es.second;
    if (ls.slot_inline[slot]) {  // fenced by the stream order; not ready when the FFN was enqueued
      ls.slot_inline[slot] = 0;
      ls.slot_pending[slot] = 0;
      st->waited += 1;
      continue;
    }
    if (!ls.slot_pending[slot]) {
      st->ready_on_time += 1;
      continue;
    }
    ls.slot_pending[slot] = 0;
    const int32_t ev = ls.slot_event[slot];
    if (std::find(waited.begin(), waited.end(), ev) != waited.end()) {
      st->waited += 1;  // covered by a wait already enqueued for this round
      continue;
    }
    const bool done1 = hipEventQuery(ls.slot_ready[ev]) == hipSuccess;
    const bool done2 = ls.slot_whole[ev] || hipEventQuery(ls.slot_ready2[ev]) == hipSuccess;
    if (done1 && done2) {
      st->ready_on_time += 1;
      continue;
    }
    if (!done1) SPP_HIP(hipStreamWaitEvent(c->compute, ls.slot_ready[ev], 0));
    if (!done2) SPP_HIP(hipStreamWaitEvent(c->compute, ls.slot_ready2[ev], 0));
    waited.push_back(ev);
    st->waited += 1;
  }
  return SPP_OK;
}

// Diagnostics of an adapter prediction made at layer l for layer l+1 (timing
// only): its Top_{K+2}(s) (s descending, lower index first; at most n) is kept
// for scoring against layer l+1's routing, and the demand count compares the
// experts of Top_M(s) not available in layer l+1 with the budget.
void record_prediction(spp_ctx* c, int32_t l, const float* s, int32_t M_max) {
  const spp_model_desc& d = c->d;
  const int32_t top = std::min(d.n, d.K + 2);
  std::vector<int32_t> idx(d.n);
  for (int32_t e = 0; e < d.n; ++e) idx[e] = e;
  std::partial_sort(idx.begin(), idx.begin() + top, idx.end(),
                    [s](int32_t a, int32_t b) { return s[a] > s[b] || (s[a] == s[b] && a < b); });
  c->pred_top.assign(idx.begin(), idx.begin() + top);
  c->pred_target = l + 1;
  const spp::SlotPolicy& nxp = *c->layers[l + 1].policy;
  const int32_t Ms[3] = {std::max(d.K / 2, 1), d.K, d.K + 2};
  for (int j = 0; j < 3; ++j) {
    int32_t missing = 0;
    for (int32_t i = 0; i < std::min(Ms[j], top); ++i) missing += nxp.slot_of(c->pred_top[i]) < 0;
    c->stats.demand_exceeds[j] += missing > std::max(M_max, 0);
    c->stats.demand_hist[j][std::min(missing, 16)] += 1;
  }
  c->stats.pred_events += 1;
}

void score_prediction(spp_ctx* c, const int32_t* T, int32_t B) {
  const spp_model_desc& d = c->d;
  const int32_t Ms[3] = {std::max(d.K / 2, 1), d.K, d.K + 2};
  for (int32_t b = 0; b < B; ++b)
    for (int j = 0; j < 3; ++j) {
      const int32_t M = std::min<int32_t>(Ms[j], static_cast<int32_t>(c->pred_top.size()));
      for (int32_t k = 0; k < d.K; ++k)
        c->stats.recall_hits[j] +=
            std::find(c->pred_top.begin(), c->pred_top.begin() + M, T[b * d.K + k]) != c->pred_top.begin() + M;
    }
  c->stats.recall_tokens += B;
}

spp_status record_extra(spp_ctx* c, TimingSet& ts) {
  if (ts.extra_used >= static_cast<int32_t>(ts.extra.size())) {
    hipEvent_t e;
    SPP_HIP(hipEventCreateWithFlags(&e, kTimingEventFlags));
    ts.extra.push_back(e);
  }
  SPP_HIP(hipEventRecord(ts.extra[ts.extra_used++], c->compute));
  return SPP_OK;
}

spp_status round_event(spp_ctx* c, size_t r, hipEvent_t* out) {
  while (c->round_done.size() <= r) {
    hipEvent_t e;
    SPP_HIP(hipEventCreateWithFlags(&e, kOrderEventFlags));
    c->round_done.push_back(e);
  }
  *out = c->round_done[r];
  return SPP_OK;
}

// Batched decode: group the (token, k) pairs by expert (ascending expert,
// ascending token, at most kGroupTokens per group) round by round, with the
// shared experts in round 0; upload the list once; per round: the round's
// copies (waiting for the previous round's FFN, whose slots they reuse), the
// compute stream's waits for them, one grouped FFN launch; then one combine.
spp_status grouped_ffn(spp_ctx* c, LayerState& ls, const int32_t* T, int32_t B,
                       const void* h_in, void* h_out, const std::vector<spp::Round>& rounds,
                       const std::vector<spp::Transfer>& loads, spp_layer_stats* st, TimingSet& ts) {
  const spp_model_desc& d = c->d;
  const int32_t BK = B * d.K;
  bool launched = false;  // the first grouped launch stamps c->t_grouped_launched
  c->t_grouped_launched = std::chrono::steady_clock::now();
  // the (token, k) pairs of each expert in pair order: a stable counting sort
  // into context scratch (pair p belongs to token p / K)
  std::vector<int32_t>& start = c->grp_start;
  std::vector<int32_t>& order = c->grp_order;
  start.assign(d.n + 1, 0);
  for (int32_t p = 0; p < BK; ++p) start[T[p] + 1] += 1;
  for (int32_t e = 0; e < d.n; ++e) start[e + 1] += start[e];
  c->grp_fill.assign(start.begin(), start.end() - 1);
  order.resize(BK);
  for (int32_t p = 0; p < BK; ++p) order[c->grp_fill[T[p]]++] = p;
  int ng = 0;
  // groups of up to kGroupTokens rows; row i of `count` is (tok(i), pair(i))
  auto add = [&](const void* blob, int32_t count, auto row) -> bool {
    for (int32_t r0 = 0; r0 < count; r0 += spp::kGroupTokens) {
      if (ng >= c->max_groups) return false;
      spp::GroupDesc& g = c->groups_host[ng++];
      g.blob = blob;
      g.m = std::min(spp::kGroupTokens, count - r0);
      for (int32_t t = 0; t < spp::kGroupTokens; ++t) {
        const bool used = t < g.m;
        const std::pair<int32_t, int32_t> tp = used ? row(r0 + t) : std::pair<int32_t, int32_t>{0, 0};
        g.tok[t] = tp.first;
        g.pair[t] = tp.second;
      }
      g.pad = 0;
    }
    return true;
  };
  std::vector<int>& rstart = c->grp_rstart;
  std::vector<int>& rcount = c->grp_rcount;
  rstart.assign(rounds.size(), 0);
  rcount.assign(rounds.size(), 0);
  int maxg = 0;
  for (size_t r = 0; r < rounds.size(); ++r) {
    rstart[r] = ng;
    for (const auto& es : rounds[r]) {
      const int32_t* rows = order.data() + start[es.first];
      const auto routed = [&](int32_t i) { return std::pair<int32_t, int32_t>{rows[i] / d.K, rows[i]}; };
      if (!add(ls.slots + static_cast<size_t>(es.second) * c->stride, start[es.first + 1] - start[es.first], routed))
        return fail(SPP_ESTATE, "group list overflow");
    }
    if (r == 0)
      for (int32_t j = 0; j < d.n_shared; ++j) {
        const auto shared = [&](int32_t b) { return std::pair<int32_t, int32_t>{b, BK + b * d.n_shared + j}; };
        if (!add(static_cast<const uint8_t*>(ls.shared) + static_cast<size_t>(j) * c->stride, B, shared))
          return fail(SPP_ESTATE, "group list overflow");
      }
    rcount[r] = ng - rstart[r];
    maxg = std::max(maxg, rcount[r]);
  }
  // unit ranges: the widest of 192 and 128 units that divides I and still
  // gives the largest round about two workgroups per compute unit, else 64.
  // Fewer ranges write fewer partial rows and stage x less often: over 128
  // Qwen-shaped experts at B = 64, 192 units (512 workgroups) took 193.7 us
  // against 198.4 for 128 (768) and 207.8 for 256 (384)
  int upw = 64;
  for (int cand : {192, 128})
    if (d.I % cand == 0 && 10L * maxg * (d.I / cand) >= 19L * c->num_cu) {
      upw = cand;
      break;
    }
  const int nsplit = (d.I + upw - 1) / upw;
  if (nsplit > c->max_nsplit) return fail(SPP_ESTATE, "unit split exceeds the partial buffer");
  for (size_t r = 0; r < rounds.size(); ++r) {
    if (r > 0) {
      hipEvent_t done;
      if (spp_status e = round_event(c, r - 1, &done)) return e;
      SPP_HIP(hipEventRecord(done, c->compute));
      std::vector<spp::Transfer> xs;
      for (const spp::Transfer& t : loads)
        if (t.round == static_cast<int32_t>(r)) xs.push_back(t);
      if (c->timing)
        if (spp_status e = record_extra(c, ts)) return e;
      if (spp_status e = issue_demand(c, ls, xs, done)) return e;
      if (spp_status e = wait_round(c, ls, rounds[r], st)) return e;
      if (c->timing)
        if (spp_status e = record_extra(c, ts)) return e;
    }
    if (rcount[r] == 0) continue;
    spp::GroupArgs ga{};
    ga.groups = c->groups_dev + rstart[r];
    ga.ngroups = rcount[r];
    ga.nsplit = nsplit;
    ga.upw = upw;
    ga.I = d.I;
    ga.D = d.D;
    ga.x = c->x_dev;
    ga.ypart = c->ypart;
    const bool first = r == 0, last = r + 1 == rounds.size();
    SPP_HIP(spp::launch_ffn_grouped(ga, c->compute, c->timing && first ? ts.ev[kEvFfnBegin] : nullptr,
                                    c->timing && last ? ts.ev[kEvFfnEnd] : nullptr));
    if (!launched) c->t_grouped_launched = std::chrono::steady_clock::now();
    launched = true;
  }
  spp::CombineBArgs cb{};
  cb.ypart = c->ypart;
  cb.gates = reinterpret_cast<const float*>(c->res_dev + c->off_gates);
  cb.B = B;
  cb.K = d.K;
  cb.n_shared = d.n_shared;
  cb.nsplit = nsplit;
  cb.D = d.D;
  cb.res_h = h_in;
  cb.res_u = d.has_proj ? c->u_dev : nullptr;
  cb.out = h_out;
  SPP_HIP(spp::launch_combine_batched(cb, d.dtype, c->compute));
  c->stats.ffn_launches += 1;
  return SPP_OK;
}

spp_status layer_forward_impl(spp_ctx* c, int32_t l, const void* h_in, void* h_out, int32_t B, int32_t M_max,
                              int32_t* topk_out, float* gate_out, spp_layer_stats* st_out) {
  if (spp_status s = check_layer(c, l, true)) return s;
  const spp_model_desc& d = c->d;
  if (!h_in || !h_out) return fail(SPP_EINVAL, "h_in / h_out is NULL");
  if (h_in == h_out) return fail(SPP_EINVAL, "h_in and h_out may not alias");
  if (B < 1 || B > d.max_batch) return fail(SPP_EINVAL, "B must be in [1, max_batch]");
  if (M_max < -1) return fail(SPP_EINVAL, "M_max must be >= -1");
  LayerState& ls = c->layers[l];
  // a prediction for layer l+1: the adapter's priorities, or (Naive Prefetch)
  // the preceding step's experts of layer l+1; the adapter runs only for the first
  const bool naive = c->prefetch_source == SPP_PREFETCH_PREV_TOKEN;
  const bool adapter_on = l < d.L - 1 && M_max >= 0 && !naive && ls.A != nullptr && d.r > 0;
  const bool predict = adapter_on || (naive && l < d.L - 1 && M_max >= 0);
  if (predict && M_max > 0 && !c->layers[l + 1].bound) return fail(SPP_ESTATE, "next layer not bound");
  const int64_t tau = ++c->clock;
  const int dt = d.dtype;
  const size_t row_bytes = static_cast<size_t>(d.D) * c->elem;

  TimingSet ts;
  if (c->timing) {
    if (spp_status s = take_set(c, &ts)) return s;
    ts.l = l;
    ts.predicted = predict;
    SPP_HIP(hipEventRecord(ts.ev[kEvStart], c->compute));
  }
  if (d.has_proj) {
    spp::ProjArgs pa{h_in, ls.proj, c->u_dev, B, d.D, d.rms_eps};
    SPP_HIP(spp::launch_proj(pa, dt, c->compute));
  }
  int32_t* topk_dev = reinterpret_cast<int32_t*>(c->res_dev);
  float* gates_dev = reinterpret_cast<float*>(c->res_dev + c->off_gates);
  float* s_dev = reinterpret_cast<float*>(c->res_dev + c->off_s);
  spp::RouterArgs ra{};
  ra.h = h_in;
  ra.u = d.has_proj ? c->u_dev : nullptr;
  ra.Wr = ls.router_w;
  ra.A = adapter_on ? ls.A : nullptr;
  ra.Bm = ls.Bm;
  ra.x_out = c->x_dev;
  ra.zbuf = c->zbuf;
  ra.ztag = c->ztag;
  ra.topk = topk_dev;
  ra.gates = gates_dev;
  ra.s = s_dev;
  ra.route_rec = c->rec_host_dev;
  ra.gate_rec = c->rec_host_dev + static_cast<size_t>(d.max_batch) * d.K;
  ra.s_rec = adapter_on ? c->rec_host_dev + 2 * static_cast<size_t>(d.max_batch) * d.K : nullptr;
  ra.counter = c->counter;
  ra.B = B;
  ra.D = d.D;
  ra.n = d.n;
  ra.K = d.K;
  ra.r = d.r;
  ra.eps = d.rms_eps;
  ra.x_given = 0;
  ra.router_on = 1;
  ra.seq = next_router_seq(c);
  SPP_HIP(spp::launch_router(ra, dt, c->compute));
  const auto t_router = std::chrono::steady_clock::now();
  if (c->timing) SPP_HIP(hipEventRecord(ts.ev[kEvRouted], c->compute));
  const bool split_ok = c->ffn_overlap && !c->grouped && B == 1;
  if (split_ok) SPP_HIP(hipEventRecord(c->route_done, c->compute));
  if (spp_status e = wait_router(c, ra.seq, 0, B)) {
    c->clock = tau - 1;
    if (c->timing) c->free_sets.push_back(ts);
    return e;
  }
  const auto t_routed = std::chrono::steady_clock::now();

  const int32_t* T = c->host_T.data();
  const float* g = c->host_g.data();
  const float* s = c->host_s.data();  // valid after the wait for kind 1
  const int32_t BK = B * d.K;
  const bool batched = c->grouped;  // the tiled layout is read by the grouped kernel only
  {
    // refusals after the routing leave the context as it was before the call
    // (the step clock included); nothing below this point has changed it yet
    spp_status bad = SPP_OK;
    std::string msg;
    for (int32_t i = 0; i < BK && bad == SPP_OK; ++i)
      if (T[i] < 0 || T[i] >= d.n) bad = SPP_EHIP, msg = "router produced an out-of-range expert id";
    if (bad == SPP_OK && !batched && ls.policy->distinct(T, BK) > d.S)
      bad = SPP_ESTATE, msg = "batch demand exceeds the slot count; more than S distinct experts per step "
                              "needs the batched bf16 path";
    if (bad != SPP_OK) {
      c->clock = tau - 1;
      if (c->timing) c->free_sets.push_back(ts);
      return fail(bad, msg);
    }
  }
  if (c->timing && c->pending_sets.size() >= 64) harvest(c, c->pending_sets.size());
  if (c->timing && c->pred_target == l) score_prediction(c, T, B);
  c->pred_target = -1;
  std::vector<float> s_naive;
  if (naive && predict) {
    // gate mass of each expert of layer l+1 at its preceding step (fp64 in
    // token order, then fp32); -inf marks the experts it did not use
    const LayerState& nl = c->layers[l + 1];
    std::vector<double> acc(d.n, -INFINITY);
    for (size_t i = 0; i < nl.prev_T.size(); ++i) {
      double& a = acc[nl.prev_T[i]];
      a = (std::isinf(a) ? 0.0 : a) + static_cast<double>(nl.prev_g[i]);
    }
    s_naive.resize(d.n);
    for (int32_t e = 0; e < d.n; ++e) s_naive[e] = static_cast<float>(acc[e]);
    s = s_naive.data();
  }

  spp_layer_stats st{};
  st.exposed_us = -1.f;
  st.layer_us = -1.f;
  {
    std::vector<char> seen(d.n, 0);
    for (int32_t i = 0; i < BK; ++i) {
      const int32_t e = T[i];
      if (seen[e]) continue;
      seen[e] = 1;
      if (ls.policy->available(e)) st.hits += 1;
    }
    for (int32_t e : ls.pending_prefetch) st.prefetch_used += seen[e] ? 1 : 0;
    for (int32_t i = 0; i < BK; ++i) st.token_hits += ls.policy->available(T[i]) ? 1 : 0;
  }
  ls.pending_prefetch.clear();
  std::string why;
  std::vector<spp::Round> rounds;
  if (!ls.policy->on_demand(T, BK, tau, &c->last_loads, &rounds, &why)) return fail(SPP_ESTATE, why);
  st.misses = static_cast<int32_t>(c->last_loads.size());

  // the compute stream's wait for expert copies starts here (on-demand loads
  // enqueued on it, or its waits for the copy streams)
  if (c->timing) SPP_HIP(hipEventRecord(ts.ev[kEvWaitA], c->compute));
  {
    std::vector<spp::Transfer> first;
    for (const spp::Transfer& t : c->last_loads)
      if (t.round == 0) first.push_back(t);
    if (c->timing) ts.shared = !first.empty() && prefetch_in_flight(c);
    if (spp_status e = issue_demand(c, ls, first, ls.last_read_valid ? ls.last_read : nullptr)) return e;
  }
  if (c->timing) SPP_HIP(hipEventRecord(ts.ev[kEvLoaded], c->compute));

  // the batch-1 FFN's work list (routed experts in T order, then the shared ones)
  auto build_ffn = [&](int32_t b, spp::FfnArgs* fa) -> int {
    *fa = spp::FfnArgs{};
    int nW = 0;
    for (int32_t k = 0; k < d.K; ++k) {
      fa->blob[nW] = ls.slots + static_cast<size_t>(ls.policy->slot_of(T[b * d.K + k])) * c->stride;
      fa->gate_idx[nW] = b * d.K + k;
      ++nW;
    }
    for (int32_t j = 0; j < d.n_shared; ++j) {
      fa->blob[nW] = static_cast<const uint8_t*>(ls.shared) + static_cast<size_t>(j) * c->stride;
      fa->gate_idx[nW] = -1;
      ++nW;
    }
    fa->nW = nW;
    fa->I = d.I;
    fa->D = d.D;
    fa->codec = d.expert_codec;
    fa->x = c->x_dev + static_cast<size_t>(b) * d.D;
    fa->gates = gates_dev;
    fa->partial = c->partial;
    // sweep order, except under the FFN split, whose two launches need every
    // workgroup on one item (the units kernel's assignment)
    if (d.expert_codec == SPP_CODEC_Q4) {
      if (!split_ok) {
        const int g = spp::ffn_grid_q4_sweep(nW * d.I, &fa->rounds, &fa->upp);
        if (g > 0) return g;
      }
      return spp::ffn_grid_q4(nW * d.I, d.I, &fa->upw, &fa->upp);
    }
    if (!split_ok) {
      const int g = spp::ffn_grid_slices(nW * d.I, d.D, d.dtype, c->ffn_wgs, &fa->rounds);
      if (g > 0) return g;
    }
    return spp::ffn_grid_for(nW * d.I, c->ffn_wgs, &fa->upw);
  };
  // FFN split (batch 1, on request): the experts whose data is complete now
  // (resident, or a finished copy) run on compute2 beside the on-demand
  // copies; the late ones (copied in this call, or still in flight) run on the
  // compute stream after their copies.  Each workgroup works on one expert, so
  // the two launches write the partial rows a single launch would write, and
  // the combine gives the same bits.
  spp::FfnArgs fa0{};
  int grid0 = 0;
  uint32_t late = 0, all_items = 0;
  bool split = false;
  if (split_ok) {
    grid0 = build_ffn(0, &fa0);
    all_items = fa0.nW >= 32 ? 0xFFFFFFFFu : ((1u << fa0.nW) - 1u);
    if (d.I % fa0.upw == 0) {
      for (int32_t k = 0; k < d.K; ++k) {
        const int32_t slot = ls.policy->slot_of(T[k]);
        bool pending = ls.slot_inline[slot] != 0;
        if (!pending && ls.slot_pending[slot]) {
          const int32_t ev = ls.slot_event[slot];
          pending = hipEventQuery(ls.slot_ready[ev]) != hipSuccess || (!ls.slot_whole[ev] && hipEventQuery(ls.slot_ready2[ev]) != hipSuccess);
        }
        if (pending) late |= 1u << k;
      }
      split = late != 0 && late != all_items;
    }
    if (split) {
      if (hipEventQuery(c->route_done) != hipSuccess) SPP_HIP(hipStreamWaitEvent(c->compute2, c->route_done, 0));
      spp::FfnArgs hits = fa0;
      hits.skip_mask = late;
      SPP_HIP(spp::launch_ffn(hits, grid0, dt, c->compute2, nullptr, nullptr));
      SPP_HIP(hipEventRecord(c->hits_done, c->compute2));
      c->stats.ffn_split_launches += 1;
    }
  }

  // RAW: the FFN reads each needed slot only after its copy completed
  if (spp_status e = wait_round(c, ls, rounds[0], &st)) return e;
  if (c->timing) SPP_HIP(hipEventRecord(ts.ev[kEvWaitB], c->compute));
  if (batched) {
    if (spp_status e = grouped_ffn(c, ls, T, B, h_in, h_out, rounds, c->last_loads, &st, ts)) return e;
  }
  std::chrono::steady_clock::time_point t_ffn{};
  for (int32_t b = 0; b < B && !batched; ++b) {
    spp::FfnArgs fa{};
    const int grid = split_ok ? grid0 : build_ffn(b, &fa);
    if (split_ok) fa = fa0;
    if (split) fa.skip_mask = all_items & ~late;
    const bool stamp = c->timing && b == B - 1;
    SPP_HIP(spp::launch_ffn(fa, grid, dt, c->compute, stamp ? ts.ev[kEvFfnBegin] : nullptr,
                            stamp ? ts.ev[kEvFfnEnd] : nullptr));
    if (b == 0) t_ffn = std::chrono::steady_clock::now();
    if (split && hipEventQuery(c->hits_done) != hipSuccess) SPP_HIP(hipStreamWaitEvent(c->compute, c->hits_done, 0));
    spp::CombineArgs ca{};
    ca.partial = c->partial;
    ca.nparts = grid;
    ca.D = d.D;
    ca.res_h = static_cast<const uint8_t*>(h_in) + b * row_bytes;
    ca.res_u = d.has_proj ? c->u_dev + static_cast<size_t>(b) * d.D : nullptr;
    ca.out = static_cast<uint8_t*>(h_out) + b * row_bytes;
    SPP_HIP(spp::launch_combine(ca, dt, c->compute));
    c->stats.ffn_launches += 1;
  }
  SPP_HIP(hipEventRecord(ls.last_read, c->compute));
  ls.last_read_valid = true;
  if (c->timing) {
    SPP_HIP(hipEventRecord(ts.ev[kEvEnd], c->compute));
    c->pending_sets.push_back(ts);
  }
  {
    if (batched) t_ffn = c->t_grouped_launched;
    const auto us = [](std::chrono::steady_clock::duration dt) {
      return std::chrono::duration<double, std::micro>(dt).count();
    };
    c->stats.host_route_us += us(t_routed - t_router);
    c->stats.host_decide_us += us(t_ffn - t_routed);
  }
  // prefetch selection for layer l+1, after the FFN launch: the adapter's
  // priorities have records of their own, which the batched selection writes
  // after every token's routing, so the FFN does not wait for them
  if (adapter_on)
    if (spp_status e = wait_router(c, ra.seq, 1, B)) return e;
  LayerState* nx = predict && M_max > 0 ? &c->layers[l + 1] : nullptr;
  c->last_pref.clear();
  c->last_s_valid = predict;
  c->last_B = B;
  c->logits_valid = !(adapter_on && B > 1);  // the batched selection overwrites logits with pi_hat
  if (adapter_on && c->timing) record_prediction(c, l, s, M_max);
  if (predict) {
    std::memcpy(c->last_s.data(), s, sizeof(float) * d.n);
    if (nx) {
      nx->policy->prefetch(s, M_max, tau, &c->last_pref);
      nx->pending_prefetch.clear();
      for (const spp::Transfer& t : c->last_pref) nx->pending_prefetch.push_back(t.expert);
      st.prefetched = static_cast<int32_t>(c->last_pref.size());
    }
    c->stats.prefetch_hist[std::min(st.prefetched, 16)] += 1;
  }

  // prefetches for layer l+1, behind every on-demand load (in copy-stream
  // order, or after the completion of the copy kernels on the compute stream)
  // and after the FFN launch (the host time they take then overlaps the FFN)
  if (nx && !c->last_pref.empty()) {
    if (spp_status e = issue_copies(c, *nx, c->last_pref, nx->last_read_valid ? nx->last_read : nullptr, false))
      return e;
    if (c->timing) {
      // marks the end of these copies on both copy streams, for the next
      // on-demand loads' question whether a prefetch still holds the link
      for (int k = 0; k < 2; ++k) SPP_HIP(hipEventRecord(c->pf_done[k], k == 0 ? c->copy : c->copy2));
      c->pf_done_valid = true;
    }
  }
  if (c->timing_level >= 2 && st_out) {
    SPP_HIP(hipEventSynchronize(ts.ev[kEvEnd]));
    double exposed = 1e3 * elapsed(ts.ev[kEvWaitA], ts.ev[kEvWaitB]);
    for (int32_t q = 0; q + 1 < ts.extra_used; q += 2) exposed += 1e3 * elapsed(ts.extra[q], ts.extra[q + 1]);
    st.exposed_us = static_cast<float>(exposed);
    st.layer_us = static_cast<float>(1e3 * elapsed(ts.ev[kEvStart], ts.ev[kEvEnd]));
  }

  if (topk_out) std::memcpy(topk_out, T, sizeof(int32_t) * BK);
  if (gate_out) std::memcpy(gate_out, g, sizeof(float) * BK);
  ls.prev_T.assign(T, T + BK);
  ls.prev_g.assign(g, g + BK);
  c->stats.layer_calls += 1;
  c->stats.hits += st.hits;
  c->stats.misses += st.misses;
  c->stats.prefetched += st.prefetched;
  c->stats.prefetch_used += st.prefetch_used;
  c->stats.ready_on_time += st.ready_on_time;
  c->stats.waited += st.waited;
  if (st_out) *st_out = st;
  return SPP_OK;
}

}  // namespace

extern "C" {

size_t spp_blob_stride(const spp_model_desc* d) {
  if (!d) return 0;
  return round_up(expert_bytes(*d), 4096);
}

int32_t spp_blob_layout(const spp_model_desc* d) {
  if (!d) return -1;
  if (d->expert_codec == SPP_CODEC_Q4) return SPP_LAYOUT_Q4_UNITS;
  return tiled_layout(*d) ? SPP_LAYOUT_TILED : SPP_LAYOUT_UNITS;
}

spp_status spp_pack_expert_q4(const spp_model_desc* d, const uint8_t* gq, const uint16_t* gs, const uint8_t* uq,
                              const uint16_t* us, const uint8_t* dq, const uint16_t* ds, void* blob) {
  std::string why;
  if (!desc_ok(d, &why)) return fail(SPP_EINVAL, why);
  if (d->expert_codec != SPP_CODEC_Q4) return fail(SPP_EINVAL, "desc does not use the 4-bit expert codec");
  if (!gq || !gs || !uq || !us || !dq || !ds || !blob) return fail(SPP_EINVAL, "a NULL pointer was passed");
  const size_t D = d->D, I = d->I, nb = D / 32, cb = D / 2, sb = nb * 2;
  const size_t unit = 3 * cb + 3 * sb;
  for (size_t k = 0; k < I * D; ++k)
    if (gq[k] > 15 || uq[k] > 15 || dq[k] > 15) return fail(SPP_EINVAL, "4-bit codes must be in 0..15");
  uint8_t* o = static_cast<uint8_t*>(blob);
  for (size_t i = 0; i < I; ++i) {
    uint8_t* u = o + i * unit;
    for (size_t j = 0; j < cb; ++j) {
      u[j] = static_cast<uint8_t>(gq[i * D + 2 * j] | (gq[i * D + 2 * j + 1] << 4));
      u[cb + j] = static_cast<uint8_t>(uq[i * D + 2 * j] | (uq[i * D + 2 * j + 1] << 4));
      u[2 * cb + j] = static_cast<uint8_t>(dq[(2 * j) * I + i] | (dq[(2 * j + 1) * I + i] << 4));
    }
    std::memcpy(u + 3 * cb, gs + i * nb, sb);
    std::memcpy(u + 3 * cb + sb, us + i * nb, sb);
    std::memcpy(u + 3 * cb + 2 * sb, ds + i * nb, sb);
  }
  const size_t bytes = expert_bytes(*d);
  std::memset(o + bytes, 0, round_up(bytes, 4096) - bytes);
  return SPP_OK;
}

spp_status spp_pack_expert(const spp_model_desc* d, const void* gate, const void* up, const void* down,
                           void* blob) {
  std::string why;
  if (!desc_ok(d, &why)) return fail(SPP_EINVAL, why);
  if (d->expert_codec != SPP_CODEC_PLAIN) return fail(SPP_EINVAL, "4-bit experts are packed by spp_pack_expert_q4");
  if (!gate || !up || !down || !blob) return fail(SPP_EINVAL, "gate, up, down and blob must not be NULL");
  const size_t D = d->D, I = d->I, es = d->dtype == SPP_DTYPE_BF16 ? 2 : 4;
  const uint8_t* g = static_cast<const uint8_t*>(gate);
  const uint8_t* u = static_cast<const uint8_t*>(up);
  const uint8_t* w = static_cast<const uint8_t*>(down);
  uint8_t* o = static_cast<uint8_t*>(blob);
  if (!tiled_layout(*d)) {
    for (size_t i = 0; i < I; ++i) {
      std::memcpy(o + (3 * i + 0) * D * es, g + i * D * es, D * es);
      std::memcpy(o + (3 * i + 1) * D * es, u + i * D * es, D * es);
      uint8_t* col = o + (3 * i + 2) * D * es;
      for (size_t r = 0; r < D; ++r) std::memcpy(col + r * es, w + (r * I + i) * es, es);
    }
  } else {
    const size_t nb = D / 256, nt = I / 16;
    const uint8_t* src[2] = {g, u};
    for (size_t t = 0; t < nt; ++t)
      for (size_t b = 0; b < nb; ++b)
        for (size_t m = 0; m < 2; ++m)
          for (size_t j = 0; j < 8; ++j)
            for (size_t l = 0; l < 64; ++l) {
              const size_t piece = (((t * nb + b) * 2 + m) * 8 + j) * 64 + l;
              const size_t row = 16 * t + (l & 15), col = 256 * b + 32 * j + 8 * (l >> 4);
              std::memcpy(o + piece * 8 * es, src[m] + (row * D + col) * es, 8 * es);
            }
    uint8_t* dn = o + 2 * I * D * es;
    for (size_t sl = 0; sl < nb; ++sl)
      for (size_t i = 0; i < I; ++i)
        for (size_t c = 0; c < 256; ++c)
          std::memcpy(dn + ((sl * I + i) * 256 + c) * es, w + ((256 * sl + c) * I + i) * es, es);
  }
  const size_t bytes = 3 * I * D * es, stride = round_up(bytes, 4096);
  std::memset(o + bytes, 0, stride - bytes);
  return SPP_OK;
}

spp_status spp_create(const spp_model_desc* desc, void* hip_stream, spp_ctx** out) {
  return create_impl(desc, hip_stream, out);
}

spp_status spp_destroy(spp_ctx* ctx) {
  if (!ctx) return fail(SPP_EINVAL, "ctx is NULL");
  free_ctx(ctx);
  return SPP_OK;
}

spp_status spp_bind_layer(spp_ctx* c, int32_t l, const void* router_w, const void* adapter_a, const void* adapter_b,
                          const void* proj_w, const void* shared_blobs, const void* host_store) {
  if (spp_status s = check_layer(c, l, false)) return s;
  const spp_model_desc& d = c->d;
  if (!router_w || !host_store) return fail(SPP_EINVAL, "router_w and host_store are required");
  if ((adapter_a == nullptr) != (adapter_b == nullptr)) return fail(SPP_EINVAL, "adapter_a and adapter_b go together");
  if (adapter_a && (l == d.L - 1 || d.r == 0)) return fail(SPP_EINVAL, "the last layer (or r == 0) has no adapter");
  if ((proj_w != nullptr) != (d.has_proj == 1)) return fail(SPP_EINVAL, "proj_w must be given iff has_proj");
  if ((shared_blobs != nullptr) != (d.n_shared > 0)) return fail(SPP_EINVAL, "shared_blobs must be given iff n_shared > 0");
  if (reinterpret_cast<uintptr_t>(host_store) % 16 != 0) return fail(SPP_EINVAL, "host_store must be 16-byte aligned");
  void* store_dev = nullptr;
  if (hipHostGetDevicePointer(&store_dev, const_cast<void*>(host_store), 0) != hipSuccess || !store_dev) {
    (void)hipGetLastError();
    return fail(SPP_EINVAL, "host_store is not pinned host memory");
  }
  LayerState& ls = c->layers[l];
  ls.host_store_dev = static_cast<const uint8_t*>(store_dev);
  ls.router_w = router_w;
  ls.A = adapter_a;
  ls.Bm = adapter_b;
  ls.proj = proj_w;
  ls.shared = shared_blobs;
  ls.host_store = static_cast<const uint8_t*>(host_store);
  ls.bound = true;
  return SPP_OK;
}

spp_status spp_set_resident(spp_ctx* c, int32_t l, const int32_t* experts, int32_t count) {
  if (spp_status s = check_layer(c, l, true)) return s;
  LayerState& ls = c->layers[l];
  spp::SlotPolicy trial(c->d.S, c->d.n);
  std::string why;
  if (!trial.set_resident(experts, count, &why)) return fail(SPP_EINVAL, why);
  if (spp_status s = sync_all(c)) return s;
  const std::vector<int32_t> before(c->d.S, spp::kEmpty);
  ls.policy->set_resident(experts, count, &why);
  ls.pending_prefetch.clear();
  ls.prev_T.clear();  // a new decode sequence: no preceding step
  ls.prev_g.clear();
  return fill_slots(c, ls, before);
}

spp_status spp_set_copy_engine(spp_ctx* c, int32_t engine) {
  if (spp_status s = check_ctx(c)) return s;
  if (engine != SPP_COPY_KERNEL && engine != SPP_COPY_SDMA && engine != SPP_COPY_SPLIT)
    return fail(SPP_EINVAL, "engine must be SPP_COPY_KERNEL, SPP_COPY_SDMA or SPP_COPY_SPLIT");
  c->copy_engine = engine;
  return SPP_OK;
}

spp_status spp_set_prefetch_source(spp_ctx* c, int32_t source) {
  if (!c) return fail(SPP_EINVAL, "ctx is NULL");
  if (source != SPP_PREFETCH_ADAPTER && source != SPP_PREFETCH_PREV_TOKEN)
    return fail(SPP_EINVAL, "source must be SPP_PREFETCH_ADAPTER or SPP_PREFETCH_PREV_TOKEN");
  c->prefetch_source = source;
  return SPP_OK;
}

spp_status spp_set_slot_table(spp_ctx* c, int32_t l, const int32_t* experts, const int64_t* stamps) {
  if (spp_status s = check_layer(c, l, true)) return s;
  if (!experts) return fail(SPP_EINVAL, "experts is NULL");
  LayerState& ls = c->layers[l];
  spp::SlotPolicy trial(c->d.S, c->d.n);
  std::string why;
  if (!trial.set_table(experts, stamps, &why)) return fail(SPP_EINVAL, why);
  if (spp_status s = sync_all(c)) return s;
  const std::vector<int32_t> before = ls.policy->slot_experts();
  ls.policy->set_table(experts, stamps, &why);
  ls.pending_prefetch.clear();
  return fill_slots(c, ls, before);
}

spp_status spp_get_slot_table(spp_ctx* c, int32_t l, int32_t* experts_out, int64_t* stamps_out) {
  if (spp_status s = check_layer(c, l, false)) return s;
  const LayerState& ls = c->layers[l];
  if (experts_out) std::memcpy(experts_out, ls.policy->slot_experts().data(), sizeof(int32_t) * c->d.S);
  if (stamps_out) std::memcpy(stamps_out, ls.policy->slot_stamps().data(), sizeof(int64_t) * c->d.S);
  return SPP_OK;
}

spp_status spp_get_clock(spp_ctx* c, int64_t* tau_out) {
  if (spp_status s = check_ctx(c)) return s;
  if (!tau_out) return fail(SPP_EINVAL, "tau_out is NULL");
  *tau_out = c->clock;
  return SPP_OK;
}

spp_status spp_set_clock(spp_ctx* c, int64_t tau) {
  if (spp_status s = check_ctx(c)) return s;
  if (tau < 0) return fail(SPP_EINVAL, "tau must be >= 0");
  c->clock = tau;
  return SPP_OK;
}

spp_status adapter_predict(spp_ctx* c, int32_t l, const float* x_dev, int32_t B, float* s_out) {
  if (spp_status s = check_layer(c, l, true)) return s;
  const spp_model_desc& d = c->d;
  LayerState& ls = c->layers[l];
  if (!x_dev || !s_out) return fail(SPP_EINVAL, "x_dev / s_out is NULL");
  if (B < 1 || B > d.max_batch) return fail(SPP_EINVAL, "B must be in [1, max_batch]");
  if (!ls.A || d.r == 0) return fail(SPP_ESTATE, "layer has no adapter");
  spp::RouterArgs ra{};
  ra.u = x_dev;
  ra.s_rec = c->rec_host_dev + 2 * static_cast<size_t>(d.max_batch) * d.K;
  ra.A = ls.A;
  ra.Bm = ls.Bm;
  ra.zbuf = c->zbuf;
  ra.ztag = c->ztag;
  ra.s = reinterpret_cast<float*>(c->res_dev + c->off_s);
  ra.counter = c->counter;
  ra.B = B;
  ra.D = d.D;
  ra.n = d.n;
  ra.K = d.K;
  ra.r = d.r;
  ra.eps = d.rms_eps;
  ra.x_given = 1;
  ra.router_on = 0;
  c->logits_valid = false;
  ra.seq = next_router_seq(c);
  SPP_HIP(spp::launch_router(ra, d.dtype, c->compute));
  if (spp_status e = wait_router(c, ra.seq, 1, B)) return e;
  std::memcpy(s_out, c->host_s.data(), sizeof(float) * d.n);
  return SPP_OK;
}

spp_status select_prefetch_budget(double window_us, double per_expert_cost_us, int32_t n_experts, int32_t* M_max_out) {
  if (!M_max_out) return fail(SPP_EINVAL, "M_max_out is NULL");
  if (!spp::prefetch_budget(window_us, per_expert_cost_us, n_experts, M_max_out))
    return fail(SPP_EINVAL, "window and cost must be finite, cost > 0, n >= 0");
  return SPP_OK;
}

spp_status expert_cache_issue_prefetch(spp_ctx* c, int32_t target_layer, const float* s_host, int32_t M_max,
                                       int32_t* issued_out, int32_t* m_out) {
  if (spp_status s = check_layer(c, target_layer, true)) return s;
  if (!s_host || !m_out || (M_max > 0 && !issued_out)) return fail(SPP_EINVAL, "s_host / issued_out / m_out is NULL");
  if (M_max < 0) return fail(SPP_EINVAL, "M_max must be >= 0");
  LayerState& ls = c->layers[target_layer];
  const int64_t tau = ++c->clock;
  std::vector<spp::Transfer> placed;
  ls.policy->prefetch(s_host, M_max, tau, &placed);
  if (spp_status e = issue_copies(c, ls, placed, ls.last_read_valid ? ls.last_read : nullptr, false)) return e;
  ls.pending_prefetch.clear();
  for (size_t i = 0; i < placed.size(); ++i) {
    issued_out[i] = placed[i].expert;
    ls.pending_prefetch.push_back(placed[i].expert);
  }
  *m_out = static_cast<int32_t>(placed.size());
  c->stats.prefetched += *m_out;
  c->stats.prefetch_hist[std::min(*m_out, 16)] += 1;
  return SPP_OK;
}

spp_status moe_layer_forward(spp_ctx* c, int32_t l, const void* h_in_dev, void* h_out_dev, int32_t B, int32_t M_max,
                             int32_t* topk_out, float* gate_out, spp_layer_stats* stats) {
  return layer_forward_impl(c, l, h_in_dev, h_out_dev, B, M_max, topk_out, gate_out, stats);
}

spp_status spp_decode_step(spp_ctx* c, const void* h_in_dev, void* h_out_dev, void* h_scratch_dev, int32_t B,
                           int32_t M_max, int32_t* topk_out, float* gate_out, spp_layer_stats* stats) {
  if (spp_status s = check_ctx(c)) return s;
  if (!h_in_dev || !h_out_dev || !h_scratch_dev) return fail(SPP_EINVAL, "h_in / h_out / h_scratch is NULL");
  if (h_in_dev == h_out_dev || h_in_dev == h_scratch_dev || h_out_dev == h_scratch_dev)
    return fail(SPP_EINVAL, "h_in, h_out and h_scratch must be distinct");
  if (B < 1 || B > c->d.max_batch) return fail(SPP_EINVAL, "B must be in [1, max_batch]");
  const int32_t L = c->d.L, BK = B * c->d.K;
  for (int32_t l = 0; l < L; ++l)
    if (!c->layers[l].bound) return fail(SPP_ESTATE, "every layer must be bound");
  // the last layer writes h_out; earlier layers alternate between the two buffers
  const void* src = h_in_dev;
  for (int32_t l = 0; l < L; ++l) {
    void* dst = ((L - 1 - l) % 2 == 0) ? h_out_dev : h_scratch_dev;
    if (spp_status s = layer_forward_impl(c, l, src, dst, B, M_max, topk_out ? topk_out + l * BK : nullptr,
                                          gate_out ? gate_out + l * BK : nullptr, stats ? stats + l : nullptr))
      return s;
    src = dst;
  }
  return SPP_OK;
}

const char* spp_last_error(void) { return g_err.c_str(); }

spp_status spp_get_last_transfers(spp_ctx* c, int32_t* loads_out, int32_t* n_loads, int32_t* pref_out,
                                  int32_t* n_pref, int32_t cap) {
  if (spp_status s = check_ctx(c)) return s;
  if (cap < 0) return fail(SPP_EINVAL, "cap must be >= 0");
  auto put = [cap](const std::vector<spp::Transfer>& xs, int32_t* out, int32_t* n) {
    if (n) *n = static_cast<int32_t>(xs.size());
    if (!out) return;
    for (size_t i = 0; i < xs.size() && static_cast<int32_t>(i) < cap; ++i) {
      out[3 * i] = xs[i].expert;
      out[3 * i + 1] = xs[i].slot;
      out[3 * i + 2] = xs[i].evicted;
    }
  };
  put(c->last_loads, loads_out, n_loads);
  put(c->last_pref, pref_out, n_pref);
  return SPP_OK;
}

spp_status spp_get_last_priorities(spp_ctx* c, float* s_out) {
  if (spp_status s = check_ctx(c)) return s;
  if (!s_out) return fail(SPP_EINVAL, "s_out is NULL");
  if (!c->last_s_valid) return fail(SPP_ESTATE, "no adapter ran in the last layer call");
  std::memcpy(s_out, c->last_s.data(), sizeof(float) * c->d.n);
  return SPP_OK;
}

spp_status spp_get_last_router_input(spp_ctx* c, float* x_out, int32_t B) {
  if (spp_status s = check_ctx(c)) return s;
  if (!x_out || B < 1 || B > c->d.max_batch) return fail(SPP_EINVAL, "bad x_out / B");
  SPP_HIP(hipStreamSynchronize(c->compute));
  SPP_HIP(hipMemcpy(x_out, c->x_dev, sizeof(float) * B * c->d.D, hipMemcpyDeviceToHost));
  return SPP_OK;
}

spp_status spp_get_last_logits(spp_ctx* c, float* z_out, int32_t B) {
  if (spp_status s = check_ctx(c)) return s;
  if (!z_out || B < 1 || B > c->last_B) return fail(SPP_EINVAL, "bad z_out / B");
  if (!c->logits_valid) return fail(SPP_ESTATE, "the last call did not leave its router logits");
  SPP_HIP(hipStreamSynchronize(c->compute));
  const size_t ldz = static_cast<size_t>(c->d.n) + c->d.r;
  SPP_HIP(hipMemcpy2D(z_out, sizeof(float) * c->d.n, c->zbuf, sizeof(float) * ldz, sizeof(float) * c->d.n, B,
                      hipMemcpyDeviceToHost));
  return SPP_OK;
}

spp_status spp_set_timing(spp_ctx* c, int32_t enabled) {
  if (spp_status s = check_ctx(c)) return s;
  if (enabled < 0 || enabled > 2) return fail(SPP_EINVAL, "timing level must be 0, 1 or 2");
  c->timing = enabled != 0;
  c->timing_level = enabled;
  return SPP_OK;
}

spp_status spp_get_layer_times(spp_ctx* c, int32_t L, int64_t* calls_out, double* exposed_us_out,
                               double* latency_us_out, int64_t* latency_calls_out) {
  if (spp_status s = check_ctx(c)) return s;
  if (L != c->d.L) return fail(SPP_EINVAL, "L must equal the context's layer count");
  if (spp_status s = sync_all(c)) return s;
  harvest(c, c->pending_sets.size());
  for (int32_t l = 0; l < L; ++l) {
    if (calls_out) calls_out[l] = c->lt_calls[l];
    if (exposed_us_out) exposed_us_out[l] = c->lt_exposed[l];
    if (latency_us_out) latency_us_out[l] = c->lt_latency[l];
    if (latency_calls_out) latency_calls_out[l] = c->lt_latency_calls[l];
  }
  return SPP_OK;
}

spp_status spp_get_run_stats(spp_ctx* c, spp_run_stats* out) {
  if (spp_status s = check_ctx(c)) return s;
  if (!out) return fail(SPP_EINVAL, "out is NULL");
  if (spp_status s = sync_all(c)) return s;
  harvest(c, c->pending_sets.size());
  *out = c->stats;
  if (c->have_prev) out->span_us += 1e3 * elapsed(c->prev.ev[kEvStart], c->prev.ev[kEvEnd]);
  return SPP_OK;
}

spp_status spp_reset_run_stats(spp_ctx* c) {
  if (spp_status s = check_ctx(c)) return s;
  if (spp_status s = sync_all(c)) return s;
  harvest(c, c->pending_sets.size());
  if (c->have_prev) {
    c->free_sets.push_back(c->prev);
    c->have_prev = false;
  }
  c->stats = spp_run_stats{};
  c->pred_target = -1;
  std::fill(c->lt_calls.begin(), c->lt_calls.end(), 0);
  std::fill(c->lt_latency_calls.begin(), c->lt_latency_calls.end(), 0);
  std::fill(c->lt_exposed.begin(), c->lt_exposed.end(), 0.0);
  std::fill(c->lt_latency.begin(), c->lt_latency.end(), 0.0);
  return SPP_OK;
}

spp_status spp_profile_expert_copy(spp_ctx* c, int32_t l, int32_t reps, double* per_expert_us) {
  if (spp_status s = check_layer(c, l, true)) return s;
  if (reps < 1 || !per_expert_us) return fail(SPP_EINVAL, "reps must be >= 1, per_expert_us non-NULL");
  if (!c->probe_dev && hipMalloc(&c->probe_dev, c->stride) != hipSuccess) return fail(SPP_ENOMEM, "probe buffer");
  LayerState& ls = c->layers[l];
  hipEvent_t e0, e1;
  SPP_HIP(hipEventCreate(&e0));
  SPP_HIP(hipEventCreate(&e1));
  SPP_HIP(copy_part(c, ls, c->probe_dev, 0, c->blob_bytes, c->copy));
  SPP_HIP(hipEventRecord(e0, c->copy));
  for (int32_t i = 0; i < reps; ++i)
    SPP_HIP(copy_part(c, ls, c->probe_dev, static_cast<size_t>(i % c->d.n) * c->stride, c->blob_bytes, c->copy));
  SPP_HIP(hipEventRecord(e1, c->copy));
  SPP_HIP(hipEventSynchronize(e1));
  *per_expert_us = 1e3 * elapsed(e0, e1) / reps;
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  return SPP_OK;
}

spp_status spp_probe_read_ceiling(spp_ctx* c, int32_t reps, double* us_out, double* gbs_out) {
  if (spp_status s = check_ctx(c)) return s;
  const spp_model_desc& d = c->d;
  if (reps < 1 || reps > 10000) return fail(SPP_EINVAL, "reps must be in [1, 10000]");
  if (d.dtype != SPP_DTYPE_BF16 || c->grouped)
    return fail(SPP_ESTATE, "the read probe needs bf16 or 4-bit experts in the batch-1 unit layout");
  spp::FfnArgs fa{};
  fa.nW = d.K;
  fa.I = d.I;
  fa.D = d.D;
  fa.codec = d.expert_codec == SPP_CODEC_Q4 ? 1 : 0;
  const int grid = fa.codec ? spp::ffn_grid_q4_sweep(d.K * d.I, &fa.rounds, &fa.upp)
                            : spp::ffn_grid_slices(d.K * d.I, d.D, d.dtype, c->ffn_wgs, &fa.rounds);
  if (grid <= 0) return fail(SPP_ESTATE, "the batch-1 FFN of this shape does not run in sweep order");
  if (spp_status e = sync_all(c)) return e;
  hipEvent_t e0, e1;
  SPP_HIP(hipEventCreate(&e0));
  SPP_HIP(hipEventCreate(&e1));
  const int64_t nslots = static_cast<int64_t>(d.L) * d.S;
  double total_ms = 0.0;
  hipError_t err = hipSuccess;
  for (int32_t it = 0; it < reps + 2 && err == hipSuccess; ++it) {
    // K slots per launch, rotating over every layer's pool so that a launch
    // rarely finds its bytes in the last-level cache
    for (int32_t k = 0; k < d.K; ++k) {
      const int64_t slot = (static_cast<int64_t>(it) * d.K + k) % nslots;
      fa.blob[k] = c->layers[slot / d.S].slots + static_cast<size_t>(slot % d.S) * c->stride;
    }
    err = spp::launch_read_probe(fa, grid, reinterpret_cast<uint32_t*>(c->partial), c->compute, e0, e1);
    if (err == hipSuccess) err = hipEventSynchronize(e1);
    float ms = 0.f;
    if (err == hipSuccess) err = hipEventElapsedTime(&ms, e0, e1);
    if (it >= 2) total_ms += ms;  // the first two launches warm the code and the TLB
  }
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  if (err != hipSuccess) return fail(SPP_EHIP, std::string("read probe: ") + hipGetErrorString(err));
  const double us = 1e3 * total_ms / reps;
  if (us_out) *us_out = us;
  if (gbs_out) *gbs_out = static_cast<double>(d.K) * c->blob_bytes / (us * 1e3);
  return SPP_OK;
}

spp_status spp_probe_stream_read(spp_ctx* c, int32_t reps, double* us_out, double* gbs_out) {
  if (spp_status s = check_ctx(c)) return s;
  const spp_model_desc& d = c->d;
  if (reps < 1 || reps > 10000) return fail(SPP_EINVAL, "reps must be in [1, 10000]");
  if (d.S < d.K) return fail(SPP_ESTATE, "the stream probe needs at least K slots per layer");
  if (spp_status e = sync_all(c)) return e;
  // K slots' worth of blob bytes, contiguous inside one layer's pool; the
  // groups of K slots rotate over every layer's pool, as the read probe's slots do
  const size_t bytes = static_cast<size_t>(d.K) * c->blob_bytes / 16 * 16;
  const int32_t per_pool = d.S / d.K;
  const int32_t groups = d.L * per_pool;
  hipEvent_t e0, e1;
  SPP_HIP(hipEventCreate(&e0));
  SPP_HIP(hipEventCreate(&e1));
  double total_ms = 0.0;
  hipError_t err = hipSuccess;
  for (int32_t it = 0; it < reps + 2 && err == hipSuccess; ++it) {
    const int32_t g = it % groups;
    const uint8_t* base = c->layers[g / per_pool].slots + static_cast<size_t>(g % per_pool) * d.K * c->stride;
    err = spp::launch_stream_probe(base, bytes, reinterpret_cast<uint32_t*>(c->partial), c->compute, e0, e1);
    if (err == hipSuccess) err = hipEventSynchronize(e1);
    float ms = 0.f;
    if (err == hipSuccess) err = hipEventElapsedTime(&ms, e0, e1);
    if (it >= 2) total_ms += ms;  // the first two launches warm the code and the TLB
  }
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  if (err != hipSuccess) return fail(SPP_EHIP, std::string("stream probe: ") + hipGetErrorString(err));
  const double us = 1e3 * total_ms / reps;
  if (us_out) *us_out = us;
  if (gbs_out) *gbs_out = static_cast<double>(bytes) / (us * 1e3);
  return SPP_OK;
}

spp_status spp_debug_set_poison(spp_ctx* c, int32_t enabled) {
  if (spp_status s = check_ctx(c)) return s;
  c->poison = enabled != 0;
  return SPP_OK;
}

spp_status spp_set_tier_delay(spp_ctx* c, int32_t delay_us) {
  if (spp_status s = spp_debug_set_copy_delay(c, delay_us)) return s;
  c->tier_serial = delay_us > 0;
  return SPP_OK;
}

spp_status spp_debug_set_copy_delay(spp_ctx* c, int32_t delay_us) {
  if (spp_status s = check_ctx(c)) return s;
  if (delay_us < 0 || delay_us > 100000) return fail(SPP_EINVAL, "delay_us must be in [0, 100000]");
  if (delay_us > 0 && c->wall_khz == 0) {
    int khz = 0;
    SPP_HIP(hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, c->device));
    if (khz <= 0) return fail(SPP_EHIP, "wall clock rate unavailable");
    c->wall_khz = static_cast<uint64_t>(khz);
  }
  c->copy_delay_us = delay_us;
  return SPP_OK;
}

spp_status spp_set_ffn_overlap(spp_ctx* c, int32_t enabled) {
  if (spp_status s = check_ctx(c)) return s;
  if (enabled != 0 && enabled != 1) return fail(SPP_EINVAL, "enabled must be 0 or 1");
  if (spp_status s = sync_all(c)) return s;
  c->ffn_overlap = enabled != 0;
  return SPP_OK;
}

spp_status spp_set_prefetch_parallel(spp_ctx* c, int32_t enabled) {
  if (spp_status s = check_ctx(c)) return s;
  if (enabled != 0 && enabled != 1) return fail(SPP_EINVAL, "enabled must be 0 or 1");
  c->prefetch_parallel = enabled != 0;
  return SPP_OK;
}

spp_status spp_set_ffn_workgroups(spp_ctx* c, int32_t wgs) {
  if (spp_status s = check_ctx(c)) return s;
  if (wgs < 1 || static_cast<size_t>(wgs) > spp::ffn_max_grid()) return fail(SPP_EINVAL, "wgs out of range");
  c->ffn_wgs = wgs;
  return SPP_OK;
}

// ------------------------------------------------------------ host policy

struct spp_slot_policy {
  spp::SlotPolicy p;
  spp_slot_policy(int32_t S, int32_t n) : p(S, n) {}
};

spp_status spp_policy_create(int32_t S, int32_t n, const int32_t* resident, int32_t count, spp_slot_policy** out) {
  if (!out || S < 1 || n < 1) return fail(SPP_EINVAL, "S, n must be >= 1 and out non-NULL");
  std::unique_ptr<spp_slot_policy> p(new (std::nothrow) spp_slot_policy(S, n));
  if (!p) return fail(SPP_ENOMEM, "host allocation failed");
  std::string why;
  if (!p->p.set_resident(resident, count, &why)) return fail(SPP_EINVAL, why);
  *out = p.release();
  return SPP_OK;
}

spp_status spp_policy_destroy(spp_slot_policy* p) {
  if (!p) return fail(SPP_EINVAL, "policy is NULL");
  delete p;
  return SPP_OK;
}

spp_status spp_policy_on_demand(spp_slot_policy* p, const int32_t* needed, int32_t count, int64_t tau,
                                int32_t* loads_out, int32_t* n_loads) {
  if (!p || (count > 0 && !needed) || count < 0 || !n_loads) return fail(SPP_EINVAL, "bad arguments");
  std::vector<spp::Transfer> loads;
  std::vector<spp::Round> rounds;
  std::string why;
  if (!p->p.on_demand(needed, count, tau, &loads, &rounds, &why)) return fail(SPP_EINVAL, why);
  *n_loads = static_cast<int32_t>(loads.size());
  for (size_t i = 0; i < loads.size() && loads_out; ++i) {
    loads_out[3 * i] = loads[i].expert;
    loads_out[3 * i + 1] = loads[i].slot;
    loads_out[3 * i + 2] = loads[i].evicted;
  }
  return SPP_OK;
}

spp_status spp_policy_prefetch(spp_slot_policy* p, const float* s, int32_t M_max, int64_t tau, int32_t* placed_out,
                               int32_t* n_placed) {
  if (!p || !s || !n_placed || M_max < 0) return fail(SPP_EINVAL, "bad arguments");
  std::vector<spp::Transfer> placed;
  p->p.prefetch(s, M_max, tau, &placed);
  *n_placed = static_cast<int32_t>(placed.size());
  for (size_t i = 0; i < placed.size() && placed_out; ++i) {
    placed_out[3 * i] = placed[i].expert;
    placed_out[3 * i + 1] = placed[i].slot;
    placed_out[3 * i + 2] = placed[i].evicted;
  }
  return SPP_OK;
}

spp_status spp_policy_get(spp_slot_policy* p, int32_t* experts_out, int64_t* stamps_out) {
  if (!p) return fail(SPP_EINVAL, "policy is NULL");
  if (experts_out) std::memcpy(experts_out, p->p.slot_experts().data(), sizeof(int32_t) * p->p.S());
  if (stamps_out) std::memcpy(stamps_out, p->p.slot_stamps().data(), sizeof(int64_t) * p->p.S());
  return SPP_OK;
}

}  // extern "C"
