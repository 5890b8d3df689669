// Host-side launchers of the decoder kernels (defined in lb_kernels.hip).
#pragma once

#include <hip/hip_runtime.h>

#include "lb_device.h"

namespace lb {

// Events recorded at the start and end of the next decode-kernel launch on this
// host thread (null: none).
void set_launch_events(hipEvent_t start, hipEvent_t stop);

hipError_t launch_build_order(int order, const int32_t* ids, const float* lp, const float* bo, int64_t count,
                              int32_t vocab, NgramTable t2, NgramTable t3, NgramTable dst, uint32_t* flags,
                              uint32_t* ctx_out, hipStream_t st);
hipError_t launch_begin(const DevParams& P, const DevState& S, int32_t B, hipStream_t st);
// The random 64-B line gather of lb_measure_gather, and the number of threads
// (= out entries) it runs for n gathers.
uint64_t gather_probe_threads(uint64_t n);
hipError_t launch_gather_probe(const void* table, uint64_t lines, uint64_t n, uint64_t seed, uint32_t* out,
                               hipStream_t st);
// args: device copy of the decoder's parameters and state.  out_hyps /
// out_scores non-null: the launch also writes the call's output (fin: the end
// of an utterance), as launch_output would.  opts: kOptPhaseTimers.  scratch:
// null (the decoder's lookup scratch) or a buffer laid out by scratch_layout.
hipError_t launch_decode(int K, const KArgs* args, const float* logits, const int32_t* lengths, int32_t B,
                         int32_t Tc, int32_t tau0, int32_t tau1, int32_t fin, int32_t* out_hyps, float* out_scores,
                         uint32_t opts, void* scratch, hipStream_t st);
hipError_t launch_fuse_select(int block, const DevParams& P, const DevState& S, const int32_t* flag, int32_t B,
                              hipStream_t st);
hipError_t launch_fuse_export(int block, const DevParams& P, const DevState& S, int32_t* words, int32_t* n_words,
                              int32_t B, hipStream_t st);
hipError_t launch_fuse_apply(int block, const DevParams& P, const DevState& S, const float* scores, int32_t B,
                             hipStream_t st);
hipError_t launch_output(int block, const DevParams& P, const DevState& S, const int32_t* lengths, int32_t B,
                         int32_t Tc, int32_t fin, int32_t* out_hyps, float* out_scores, hipStream_t st);

// Capacity of the per-device static lookup scratch, and its device address on
// the current device (looked up once per device).
constexpr size_t kStaticScratchBytes = size_t{64} << 20;
constexpr int kMaxDevices = 64;
hipError_t static_scratch_address(void** out);

}  // namespace lb
