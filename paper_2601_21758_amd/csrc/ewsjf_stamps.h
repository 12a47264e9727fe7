// Phase timestamps for the instrumented build (compiled with -DEWSJF_STAMPS
// into libewsjf_stamps.so; paper_2601_21758_amd/phase_stamps.py reads them).
// Thread 0 of workgroup (x < kStampBlocks, y == 0) of a kernel records the
// device's constant 100 MHz clock at numbered points of the kernel.  In the
// regular build EWSJF_STAMP expands to nothing.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ewsjf {

constexpr int kStampKernels = 4;
constexpr int kStampBlocks = 256;
constexpr int kStampPhases = 8;
constexpr int kStampSlots = kStampKernels * kStampBlocks * kStampPhases;

// Kernel ids of the stamps.
enum { kStampLocal = 0, kStampMergeRank = 1, kStampMergeExact = 2, kStampMulti = 3 };

}  // namespace ewsjf

#ifdef EWSJF_STAMPS
namespace ewsjf {
// One copy per translation unit that includes this header (no relocatable
// device code): the select kernels' unit owns the one that is read.
static __device__ uint64_t g_stamps[kStampSlots];
// The workgroup's stamps are kept in LDS while the kernel runs and written
// out at its exits (EWSJF_STAMP_FLUSH): a global store per stamp would be
// waited for by the next barrier (its release), which would lengthen the
// phase being timed.
static __shared__ uint64_t s_stamps[kStampKernels][kStampPhases];
}  // namespace ewsjf
#define EWSJF_STAMP_ON (threadIdx.x == 0 && blockIdx.y == 0 && blockIdx.x < (unsigned)::ewsjf::kStampBlocks)
// Point 0 also clears the kernel's other points (a point not reached reads 0).
#define EWSJF_STAMP(kid, phase)                                                                     \
  do {                                                                                              \
    if (EWSJF_STAMP_ON) {                                                                           \
      if ((phase) == 0)                                                                             \
        for (int ewsjf_i_ = 1; ewsjf_i_ < ::ewsjf::kStampPhases; ++ewsjf_i_)                        \
          ::ewsjf::s_stamps[(kid)][ewsjf_i_] = 0ull;                                                \
      ::ewsjf::s_stamps[(kid)][(phase)] = __builtin_amdgcn_s_memrealtime();                         \
    }                                                                                               \
  } while (0)
// A value in place of a time (read back as is).
#define EWSJF_STAMP_VALUE(kid, phase, value)                                                        \
  do {                                                                                              \
    if (EWSJF_STAMP_ON) ::ewsjf::s_stamps[(kid)][(phase)] = (uint64_t)(value);                      \
  } while (0)
// The time once `dep` (a 32-bit value of the wave) has been computed: the
// value is handed to an empty asm statement before the clock is read.
#define EWSJF_STAMP_AFTER(kid, phase, dep)                                                          \
  do {                                                                                              \
    const int ewsjf_dep_ = __builtin_amdgcn_readfirstlane((int)(dep));                              \
    asm volatile("" ::"s"(ewsjf_dep_));                                                             \
    EWSJF_STAMP(kid, phase);                                                                        \
  } while (0)
// At every exit of a stamped kernel: the workgroup's points to the device array.
#define EWSJF_STAMP_FLUSH(kid)                                                                      \
  do {                                                                                              \
    if (EWSJF_STAMP_ON)                                                                             \
      for (int ewsjf_i_ = 0; ewsjf_i_ < ::ewsjf::kStampPhases; ++ewsjf_i_)                          \
        ::ewsjf::g_stamps[((kid) * ::ewsjf::kStampBlocks + blockIdx.x) * ::ewsjf::kStampPhases +    \
                          ewsjf_i_] = ::ewsjf::s_stamps[(kid)][ewsjf_i_];                           \
  } while (0)
#else
#define EWSJF_STAMP(kid, phase) \
  do {                          \
  } while (0)
#define EWSJF_STAMP_VALUE(kid, phase, value) \
  do {                                       \
  } while (0)
#define EWSJF_STAMP_AFTER(kid, phase, dep) \
  do {                                     \
  } while (0)
#define EWSJF_STAMP_FLUSH(kid) \
  do {                         \
  } while (0)
#endif
