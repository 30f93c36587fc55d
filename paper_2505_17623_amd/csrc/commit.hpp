// commit.hpp -- launchers of the commitment kernels (commit.hip).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ra {

constexpr int kMsmChunks = 256;  // workgroups per window of the bucket method (each a chunk of the values)

// Generators first .. first + count - 1 of `domain` (32 bytes), affine, 16
// little-endian uint32 limbs each (x then y); *err set if a counter runs out.
void launch_commit_generators(const uint8_t *domain, uint64_t first, uint64_t count, uint32_t *gens, uint32_t *err,
                              hipStream_t st);

// Scalars: int16, uint16, int32 or uint64 values (kind 0..3).
int msm_windows(int kind);  // 8-bit windows of the magnitudes
size_t msm_workspace_bytes(int kind);
// sum_i v_i G_i, written as 64 big-endian bytes (x, y; zeros for the identity) to out (device)
void launch_commit(const void *vals, int kind, uint64_t n, const uint32_t *gens, void *ws, uint8_t *out,
                   hipStream_t st);

// Several tables at once: table t (values vals[t], kind kinds[t], ns[t]
// values, generators from gens[0]) uses the workspace at ws + offset t of
// msm_batch_offsets and writes its 64 bytes to out + 64 t.  The bucket passes
// run table by table; the bucket sums, bit sums and final chains of all
// tables each run in one launch.
constexpr int kCommitBatchMax = 64;
size_t msm_batch_offsets(const int *kinds, int count, size_t *offs);  // fills offs[count], returns the total
void launch_commit_batch(const void *const *vals, const int *kinds, const uint64_t *ns, int count,
                         const uint32_t *gens, void *ws, uint8_t *out, hipStream_t st);

}  // namespace ra
