// Phase stamps of the stamping build (compiled with -DCS_PHASE_STAMPS into
// libcs_stamps.so, used by the benchmark's phase report): at the end of each
// phase of a layer kernel, thread 0 of the workgroup adds the constant-rate
// wall clock to that phase's slot of a device array, and at the start of a
// unit of work (a workgroup of the chain, a tile of the table-block kernel)
// one to its count slot.  The difference of two slots' sums divided by the
// count is the mean time between the two points; stamps taken after a
// workgroup barrier time the whole workgroup, the others its first
// wavefront.  In the product build the macros expand to nothing.
//
// Slots: the one-kernel keyword-spotting chain 0 start, 1 conv1 staged,
// 2 conv1 products, 3 conv1 k-WTA, 4 conv1 lists out, 5 conv2 staged,
// 6 conv2 products, 7 conv2 pool + k-WTA + lists, 8 linear1 staged,
// 9 linear1 products, 10 linear1 sums, 11 linear1 threshold, 12 linear1
// lists, 13 end (output layer), 15 count; the table-block kernel 16 tile
// start, 17 products, 18 epilogue, 31 count, in its k-WTA on the lanes' own
// columns 19 threshold search, 20 winner masks, and 21 the time of a tile
// spent in the table blocks' products (measured per block with CS_CLOCK, added
// once per tile: an atomic per block would itself take part of the time).
#pragma once

#ifdef CS_PHASE_STAMPS
__device__ unsigned long long cs_phase_acc[32];
#define CS_STAMP(i)                                                                      \
  do {                                                                                  \
    if (threadIdx.x == 0) atomicAdd(&cs_phase_acc[(i)], (unsigned long long)wall_clock64()); \
  } while (0)
#define CS_STAMP_COUNT(i)                                                                \
  do {                                                                                  \
    if (threadIdx.x == 0) atomicAdd(&cs_phase_acc[(i)], 1ull);                          \
  } while (0)
#define CS_CLOCK() ((unsigned long long)wall_clock64())
#define CS_STAMP_ADD(i, v)                                                               \
  do {                                                                                  \
    if (threadIdx.x == 0) atomicAdd(&cs_phase_acc[(i)], (unsigned long long)(v));       \
  } while (0)
#else
#define CS_STAMP(i) \
  do {              \
  } while (0)
#define CS_STAMP_COUNT(i) \
  do {                    \
  } while (0)
#define CS_CLOCK() 0ull
#define CS_STAMP_ADD(i, v) \
  do {                     \
  } while (0)
#endif
