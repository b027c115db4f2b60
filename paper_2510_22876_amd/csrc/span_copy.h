// Device helpers shared by the kernels that move bf16 cache columns: 16-byte
// vector loads/stores with optional nontemporal hints, scalar loads of
// per-launch invariants, and the split-piece column move used for every
// out-of-place rewrite of a span (realignment and batch gathering).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace specdec {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <bool kNt>
__device__ __forceinline__ u32x4 ld16(const u32x4* p) {
  if constexpr (kNt) return __builtin_nontemporal_load(p);
  else return *p;
}

// Stores one 16-byte vector at wave_base[lane_vec].  With kNt the store is
// nontemporal and device-coherent (cache policy "nt sc1"): the line is
// written through the XCD's L2 instead of staying dirty in it until eviction
// or the end of the kernel.  Measured on MI355X against a nontemporal store
// alone: about 1% faster for the out-of-place moves and 1.4-5% for the
// in-place walk; the compiler's nontemporal store sets "nt" alone, and the
// buffer-store builtin that takes the policy bits measured 0.5-1.5% slower
// than this global store on the out-of-place moves.
//
// The store is inline assembly, so the compiler sees neither its memory
// operation nor its data registers:
//  * Wait counters: the compiler does not count it, so any wait it places
//    for a later load also covers the store (waits only get stricter); no
//    kernel here reads what another thread of the same launch stored.
//  * Hazard: on gfx950 a VALU write of the data registers of a store wider
//    than 8 bytes must come at least two wait states after the store, or the
//    store may write the new value.  The compiler inserts these for its own
//    stores; for this one the statement carries them ("s_nop 1").  With no
//    wait state the compiler once placed a 64-bit register move into the low
//    half of a zero store's data registers one instruction after it, and a
//    padding column received 8 bytes of that value.
template <bool kNt>
__device__ __forceinline__ void st16_at(u32x4* wave_base, uint32_t lane_vec, u32x4 v) {
  if constexpr (kNt)
    asm volatile("global_store_dwordx4 %0, %1, off nt sc1\n\ts_nop 1" : : "v"(wave_base + lane_vec), "v"(v) : "memory");
  else wave_base[lane_vec] = v;
}

// Index of the calling thread's wavefront in its workgroup, as a value the
// compiler knows to be uniform across the wave.
__device__ __forceinline__ int wave_index() { return __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6)); }

// Loads a value that no kernel of this launch writes, through the constant
// address space: a wave-uniform address then becomes a scalar load on the
// scalar cache path instead of a vector load queued behind the data traffic.
__device__ __forceinline__ int32_t load_invariant(const int32_t* p) {
  return *(const __attribute__((address_space(4))) int32_t*)p;
}

// One workgroup's share of an out-of-place span rewrite.  The output span has
// `total` 16-byte vectors: [0, zero_end) become +0.0, vector u in
// [zero_end, total) receives source vector u - shift.  The workgroup moves
// kPieces pieces of kTpb vectors (one per lane) starting at `base`, the
// pieces kSplit vectors apart.  Each piece is padding (stores only), content
// (one load and one store per lane), or the boundary / ragged end, where the
// source index is clamped into the kept range so every load is in bounds.  A
// span with no kept vector (zero_end >= total) is padding throughout and
// loads nothing.  `base` may be negative (a span tiled from the group
// boundary below its start, see split_misalign): vectors before the span are
// neither loaded nor stored.
template <int kPieces, int kTpb, int kSplit, int kNt>
__device__ __forceinline__ void split_pieces(const u32x4* s, u32x4* d, int64_t base, int64_t total,
                                             int64_t zero_end, int64_t shift) {
  const int t = threadIdx.x;
  const u32x4 zero = {0u, 0u, 0u, 0u};
  const int64_t lo = zero_end - shift, hi = total - 1 - shift;   // kept source range
  u32x4 v[kPieces];
#pragma unroll
  for (int j = 0; j < kPieces; ++j) {
    const int64_t p0 = base + static_cast<int64_t>(j) * kSplit;  // first vector of the piece
    if (p0 >= zero_end && p0 + kTpb <= total) {
      v[j] = ld16<(kNt & 1) != 0>(s + (p0 + t - shift));
    } else if (p0 + kTpb > zero_end && p0 < total && zero_end < total) {
      int64_t si = p0 + t - shift;
      si = si < lo ? lo : (si > hi ? hi : si);
      v[j] = ld16<(kNt & 1) != 0>(s + si);
    } else {
      v[j] = zero;
    }
  }
  // every load has landed before the first store is issued, so no store
  // waits behind another one (stores count in the same wait counter)
#pragma unroll
  for (int j = 0; j < kPieces; ++j) asm volatile("" ::"v"(v[j].x), "v"(v[j].y), "v"(v[j].z), "v"(v[j].w));
#pragma unroll
  for (int j = 0; j < kPieces; ++j) {
    const int64_t p0 = base + static_cast<int64_t>(j) * kSplit;   // the piece's first vector (wave-uniform)
    if (p0 >= total) break;
    const int64_t u = p0 + t;
    if (u >= 0 && u < total) st16_at<(kNt & 2) != 0>(d + p0, t, u >= zero_end ? v[j] : zero);
  }
}

// First vector of workgroup `sub` of a span in the split-piece layout.
template <int kPieces, int kTpb, int kSplit>
__device__ __forceinline__ int64_t split_base(uint32_t sub) {
  static_assert(kSplit % kTpb == 0, "a group is a whole number of workgroups");
  constexpr uint32_t kPerGroup = kSplit / kTpb;
  const uint32_t grp = sub / kPerGroup;
  return static_cast<int64_t>(grp) * (kPieces * kSplit) + static_cast<int64_t>(sub - grp * kPerGroup) * kTpb;
}

// Workgroups per span in the split-piece layout for spans of `vecs` vectors;
// with `misaligned`, room for one more group (a span tiled from the group
// boundary below its start).
template <int kPieces, int kTpb, int kSplit>
constexpr int64_t split_blocks(int64_t vecs, bool misaligned = false) {
  constexpr int64_t kGroup = static_cast<int64_t>(kPieces) * kSplit;
  return ((vecs + (misaligned ? kGroup - 1 : 0) + kGroup - 1) / kGroup) * (kSplit / kTpb);
}

// Output spans are tiled in groups of kPieces*kSplit vectors.  When a span
// does not start on a group boundary of the address space (a capacity that is
// not a multiple of the group), the tiling starts at the boundary below the
// span instead: every piece then covers the same aligned 1 KB slots of memory
// whatever the capacity, which keeps the stores of a group on whole aligned
// 16 KB blocks (measured on MI355X: about 8% more bandwidth than tiling from
// a 256-byte-aligned span start).  Returns the span start's offset, in
// vectors, from that boundary.
template <int kPieces, int kSplit>
__device__ __forceinline__ int64_t split_misalign(const u32x4* d) {
  constexpr uint64_t kGroup = static_cast<uint64_t>(kPieces) * kSplit;
  static_assert((kGroup & (kGroup - 1)) == 0, "the group is a power of two vectors");
  return static_cast<int64_t>((reinterpret_cast<uintptr_t>(d) / 16u) & (kGroup - 1));
}

// True when every span of a buffer (base pointer, span stride in vectors)
// starts on a group boundary, so no span needs the extra group.
template <int kPieces, int kSplit>
inline bool split_spans_aligned(const void* base, int64_t span_vecs) {
  constexpr uint64_t kGroup = static_cast<uint64_t>(kPieces) * kSplit;
  return (reinterpret_cast<uintptr_t>(base) % (kGroup * 16u)) == 0 &&
         (static_cast<uint64_t>(span_vecs) % kGroup) == 0;
}

}  // namespace specdec
