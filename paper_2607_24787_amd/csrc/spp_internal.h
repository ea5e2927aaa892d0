// Internal interface between the runtime (spp_runtime.cpp) and the gfx950
// kernels (spp_kernels.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstdint>

#include "spp.h"

namespace spp {

// Sets the calling thread's spp_last_error message and returns `s`.
spp_status set_error(spp_status s, const char* msg);

constexpr int kMaxWork = 32;       // expert blobs one FFN launch can combine
constexpr int kMaxExpertsTopK = 1024;

// Router + adapter (one launch).  Rows [0, n) are router logits (if
// router_on), rows [n, n+r) adapter hidden units (if A != nullptr).
struct RouterArgs {
  const void* h;        // [B, D] storage dtype; layer input when u == nullptr
  const float* u;       // [B, D] fp32 input (prologue output, or x itself when x_given)
  const void* Wr;       // [n, D]
  const void* A;        // [r, D] or nullptr
  const void* Bm;       // [n, r]
  float* x_out;         // [B, D] router input written by block 0 (nullptr: skip)
  float* zbuf;          // [B, n + r] logits then adapter hidden units
  uint64_t* ztag;       // [n + r] the same values tagged (seq << 32) | fp32 bits, for the batch-1
                        // single-wave tails (polled instead of a completion counter), or nullptr
  int32_t* topk;        // [B, K]
  float* gates;         // [B, K]
  float* s;             // [n]
  // host records (pinned, host-mapped; device-visible addresses) or nullptr:
  // 8-byte words (seq << 32) | payload, each written by one store, so the
  // host knows a record is this launch's when its high half equals seq
  uint64_t* route_rec;  // [B*K]: expert id of (b, k)
  uint64_t* gate_rec;   // [B*K]: gate of (b, k) (fp32 bits); a separate array, so that the K
                        // records of a token are one contiguous store per wave, not K
  uint64_t* s_rec;      // [n]: priority s_e (fp32 bits)
  unsigned* counter;    // [2] zero between launches (router rows, adapter rows)
  unsigned seq;         // this launch's sequence number (never 0)
  int B, D, n, K, r;
  float eps;
  int x_given;          // u holds x (no normalisation)
  int router_on;
};

struct FfnArgs {
  const void* blob[kMaxWork];  // expert blobs (slot or shared expert)
  int32_t gate_idx[kMaxWork];  // index into gates, or -1 for weight 1
  int nW;
  int I, D;
  int upw;                     // units per workgroup
  int upp;                     // 4-bit experts: units per wave and pass (3 or 4)
  uint32_t skip_mask;          // bit d set: work item d is left to another launch (0: run all).  A
                               // workgroup whose units belong to a skipped item writes nothing; a
                               // nonzero mask needs upw to divide I (each workgroup on one item)
  int codec;                   // 0: experts in dtype; 1: 4-bit blocks (dtype bf16)
  int rounds;                  // 0: workgroup b takes units [b*upw, (b+1)*upw) (ffn_units_kernel, and
                               // ffn_q4_kernel by range); 1..3: sweep rounds of ffn_slices_kernel (see
                               // ffn_grid_slices); 4-bit experts: 1..2 sweep passes of ffn_q4_kernel
                               // (see ffn_grid_q4_sweep); upw unused in sweep order
  const float* x;              // [D] router input of the token
  const float* gates;
  float* partial;              // [gridDim.x, D]
};

// Batched decode: one group = up to kGroupTokens tokens that share one expert.
constexpr int kGroupTokens = 16;
struct GroupDesc {
  const void* blob;                // expert blob (slot or shared expert)
  int32_t m;                       // tokens in the group, 1..kGroupTokens
  int32_t tok[kGroupTokens];       // token index b of each row
  int32_t pair[kGroupTokens];      // output pair: b*K + k (routed) or B*K + b*n_shared + j (shared)
  int32_t pad;
};

struct GroupArgs {
  const GroupDesc* groups;  // [ngroups] (device-visible; host-mapped pinned memory)
  int ngroups, nsplit, upw; // each group's I units are split into nsplit ranges of upw units
  int I, D;
  const float* x;           // [B, D] router inputs
  float* ypart;             // [npairs * nsplit, D] partial expert outputs
};

struct CombineBArgs {
  const float* ypart;       // [npairs * nsplit, D]
  const float* gates;       // [B, K]
  int B, K, n_shared, nsplit, D;
  const void* res_h;        // [B, D] residual in storage dtype (used when res_u == nullptr)
  const float* res_u;       // [B, D] fp32 residual (prologue output)
  void* out;                // [B, D] storage dtype
};

struct CombineArgs {
  const float* partial;  // [nparts, D]
  int nparts, D;
  const void* res_h;     // residual in storage dtype (used when res_u == nullptr)
  const float* res_u;    // fp32 residual (prologue output)
  void* out;             // [D] storage dtype
};

struct ProjArgs {
  const void* h;   // [B, D]
  const void* P;   // [D, D]
  float* u;        // [B, D]
  int B, D;
  float eps;
};

hipError_t launch_router(const RouterArgs& a, int dtype, hipStream_t st);
// start/stop (nullable) are stamped with the kernel's own begin/end times.
hipError_t launch_ffn(const FfnArgs& a, int grid, int dtype, hipStream_t st, hipEvent_t start, hipEvent_t stop);
hipError_t launch_combine(const CombineArgs& a, int dtype, hipStream_t st);
hipError_t launch_proj(const ProjArgs& a, int dtype, hipStream_t st);
// Grouped (batched) routed-expert FFN, bf16 only; D % 256 == 0.
hipError_t launch_ffn_grouped(const GroupArgs& a, hipStream_t st, hipEvent_t start, hipEvent_t stop);
hipError_t launch_combine_batched(const CombineBArgs& a, int dtype, hipStream_t st);
// Host-to-device copies by a copy kernel: n copies of n16 16-byte chunks each,
// from pinned host memory (its device-visible, 16-byte aligned address) to
// 16-byte aligned device memory, one after the other in one launch of `wgs`
// workgroups.
constexpr int kMaxCopyList = 32;
struct CopyList {
  const void* src[kMaxCopyList];
  void* dst[kMaxCopyList];
  int32_t n;
  uint64_t n16;
};
hipError_t launch_h2d_copies(const CopyList& list, int wgs, hipStream_t st);
hipError_t launch_spin(uint64_t ticks, uint32_t max_iter, hipStream_t st);
// Batch-1 FFN launch over `nunits` (expert, unit) pairs: units per workgroup
// (*upw) so that about `target_wgs` workgroups share the work; returns the grid.
int ffn_grid_for(int nunits, int target_wgs, int* upw);
// The same work list in sweep rounds (bf16/fp32 experts, no skip mask): the
// number of rounds (*rounds, 1..3) that puts the grid nearest `target_wgs`
// workgroups; returns the grid, or 0 when it would exceed ffn_max_grid().
int ffn_grid_slices(int nunits, int D, int dtype, int target_wgs, int* rounds);
// 4-bit experts in sweep order (no skip mask): passes (*rounds, 1 or 2) of 3
// units per wave (*upp); returns the grid, or 0 when it would exceed
// ffn_max_grid().
int ffn_grid_q4_sweep(int nunits, int* rounds, int* upp);
// The loads of a bf16 ffn_slices_kernel launch with the same arguments and
// grid, and nothing else (a read-ceiling probe); one checksum word per
// workgroup into sink [grid]; start/stop stamped with the kernel's own times.
// Plain streaming read of `bytes` (a multiple of 16) from base (16-byte
// aligned), timed by start/stop; sink takes at least 256 words.
hipError_t launch_stream_probe(const void* base, size_t bytes, uint32_t* sink, hipStream_t st, hipEvent_t start,
                               hipEvent_t stop);
hipError_t launch_read_probe(const FfnArgs& a, int grid, uint32_t* sink, hipStream_t st, hipEvent_t start,
                             hipEvent_t stop);
// 4-bit experts: whole passes of kFfnWaves * upp units per workgroup (upp 3
// or 4 units per wave and pass), as many as keep the grid near 256 workgroups.
int ffn_grid_q4(int nunits, int I, int* upw, int* upp);
size_t ffn_max_grid();

}  // namespace spp
