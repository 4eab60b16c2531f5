// Host-side arguments of the prefill and decode work items, shared by the
// kernels that run them: the prefill kernel, the decode kernel and the mixed
// prefill + decode kernel.
#pragma once

#include "decode_impl.hpp"
#include "launch.hpp"
#include "prefill_impl.hpp"

namespace ckv {

// Arguments of a prefill launch (row tiles, key partitions, workspace
// pointers); hipErrorInvalidConfiguration when the row tiles exceed a grid
// dimension.
hipError_t prefill_args(const PoolView &p, const BatchView &b, const void *q, int h_q, float scale,
                        int window, void *out, void *ws, pf::PrefillArgs &a);
// Merge of a prefill's key partitions (a.splits > 1).
hipError_t launch_prefill_merge(const pf::PrefillArgs &a, int d, int total_q, hipStream_t s);

// Arguments of a decode launch (partition length and count, head chunks,
// workspace pointers).
void decode_args(const PoolView &p, const BatchView &b, const void *q, int h_q, float scale,
                 int window, int split_len, void *out, void *ws, dc::DecodeArgs &a);
// Merge of a decode's split-K partitions (a.max_splits > 1).
hipError_t launch_decode_merge(const dc::DecodeArgs &a, int d, int num_seqs, hipStream_t s);

}  // namespace ckv
