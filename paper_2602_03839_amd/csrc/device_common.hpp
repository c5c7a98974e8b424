// device_common.hpp -- gfx950 building blocks shared by the libpulse kernels.
//
//  * FP32 -> BF16 round-to-nearest-even on the conversion unit;
//  * wave64 scans and reductions;
//  * the single-pass ordered scan across workgroups ("decoupled look-back",
//    Merrill & Garland, NVIDIA tech report NVR-2016-002), written for CDNA:
//    tiles are numbered by an atomic ticket so every tile's predecessors are
//    already resident, and each tile publishes one self-contained 64-bit
//    status word, so no fences are needed between a flag and its value.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

namespace pulse {

// ---------------------------------------------------------------- workspace
//
// The header holds three words, each on its own 128-byte cache line so that
// polls of one never contend with the atomics on another:
// word kWordTicket: ticket counter = (G0 << 24) | c, where c counts the chunks
//         of kChunk consecutive tiles drawn in the current launch and G0 is the
//         global sequence number of that launch's first tile.  Blocks are
//         persistent and draw chunks until they get one past the launch's last
//         tile.  A single device-wide counter sustains only ~75M atomics/s on
//         MI355X, so tiles are handed out kChunk at a time.
// word kWordGaveUp: set to 1 if a look-back ever gave up waiting (see look_back).
// word kWordDone: number of blocks of the current launch that have finished.
//         The last block out (every other block has made its final draw before
//         it counted itself out) stores ((G0 + ntiles) << 24) into the ticket
//         counter and 0 here, so the next launch starts at c = 0 with no reset
//         kernel.
// words kStatusOffsetWords ..: a ring of kSlots status words.  Tile with global
//         sequence g uses slot g mod kSlots and tags its word with (g / kSlots)
//         mod 256.  Every sequence number is published exactly once, in order
//         of use, so a slot holds either the current lap's word or the previous
//         lap's, whose tag differs; a stale word reads as "not ready".  A slot
//         is reused only kSlots sequence numbers later; since at most R <= 8192
//         sequence numbers are in flight at once (tiles, or two per tile for a
//         kernel that chains two scans per tile) and a look-back reaches at
//         most R of them, kSlots > 2R + 2 ensures a word is never overwritten
//         while a reader still needs it.
constexpr int kWordTicket = 0;
constexpr int kWordGaveUp = 16;
constexpr int kWordDone = 32;
constexpr int kTicketBits = 24;
constexpr uint64_t kTicketMask = (1ull << kTicketBits) - 1;
constexpr uint64_t kSeqMask = (1ull << 40) - 1;  // G0 is kept modulo 2^40
constexpr int kSlotBits = 16;
constexpr uint64_t kSlots = 1ull << kSlotBits;
constexpr int kStatusOffsetWords = 64;            // 512-byte header
constexpr size_t kWorkspaceBytes = (kStatusOffsetWords + kSlots) * sizeof(uint64_t);
constexpr uint32_t kMaxTilesPerLaunch = (1u << kTicketBits) - 1;  // < kNoTicket
// Largest grid of a ticketed launch.
constexpr uint32_t kMaxGrid = 1u << 16;

// status word: [63:62] flag, [61:54] lap tag, [53:0] value
constexpr uint64_t kFlagAggregate = 1;  // value = this tile's own count
constexpr uint64_t kFlagPrefix = 2;     // value = inclusive prefix (count_in + tiles 0..t)
constexpr uint64_t kValueMask = (1ull << 54) - 1;

// A predecessor is always resident or finished, so a look-back normally waits
// microseconds.  Only a workspace that was not zero-filled can make a tile
// wait for one that never runs; after this many polls (well under a second)
// the wave stops waiting, counts the missing tiles as empty and raises word
// kWordGaveUp of the workspace, after which no wave of the device waits any
// more: a misuse yields a wrong patch and a raised flag instead of a hung GPU.
// The flag stays raised until the workspace is zero-filled again, and
// pulse_workspace_status reports it to the host.
constexpr uint32_t kMaxPolls = 1u << 18;

// Look-back window: 64 * kLookK predecessors read at once.
constexpr int kLookK = 1;

__device__ __forceinline__ uint64_t status_word(uint64_t flag, uint64_t g, uint64_t value) {
  return (flag << 62) | (((g >> kSlotBits) & 0xFFull) << 54) | (value & kValueMask);
}

__device__ __forceinline__ uint64_t* status_slot(uint64_t* ws, uint64_t g) {
  return ws + kStatusOffsetWords + (g & (kSlots - 1));
}

__device__ __forceinline__ void status_publish(uint64_t* ws, uint64_t g, uint64_t flag,
                                               uint64_t value) {
  __hip_atomic_store(status_slot(ws, g), status_word(flag, g, value), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------- BF16 RNE
//
// FP32 -> BF16 with round-to-nearest-even, two elements at a time, on the
// gfx950 conversion unit (v_cvt_pk_bf16_f32).  With the IEEE denormal mode
// these kernels run in, it computes exactly the reference rounding: the
// nearest BF16 value, ties to the even mantissa, overflow to +-inf,
// subnormals kept, and a NaN made quiet with its sign and leading payload
// bits kept.  The exhaustive cast test compares it with the CPU reference on
// all 2^32 FP32 patterns.
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// BF16 bits of the FP32 patterns lo (bits 15:0) and hi (bits 31:16).
__device__ __forceinline__ uint32_t bf16x2_rne(uint32_t lo, uint32_t hi) {
  const f32x2_t v = {__uint_as_float(lo), __uint_as_float(hi)};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

// Change mask of two packed BF16 pairs: bit 0 = low halves differ, bit 1 =
// high halves differ (bitwise, so +0 and -0 differ and equal NaN bits match).
__device__ __forceinline__ uint32_t diff2(uint32_t a, uint32_t b) {
  const uint32_t d = a ^ b;
  return (uint32_t)((d & 0xFFFFu) != 0u) | ((uint32_t)((d >> 16) != 0u) << 1);
}

// ---------------------------------------------------------------- wave64 helpers

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// Lane move with a DPP pattern; lanes without a source (or outside the enabled
// rows) read 0.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp_or_zero(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, ROW_MASK, 0xF, false);
}

// Inclusive prefix sum over the 64 lanes of a wave, without LDS: shifts by
// 1, 2, 4, 8 inside each 16-lane row, then the row totals are carried across
// rows by the row_bcast:15 and row_bcast:31 patterns.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
  v += dpp_or_zero<0x111, 0xF>(v);  // row_shr:1
  v += dpp_or_zero<0x112, 0xF>(v);  // row_shr:2
  v += dpp_or_zero<0x114, 0xF>(v);  // row_shr:4
  v += dpp_or_zero<0x118, 0xF>(v);  // row_shr:8
  v += dpp_or_zero<0x142, 0xA>(v);  // row_bcast:15 into rows 1 and 3
  v += dpp_or_zero<0x143, 0xC>(v);  // row_bcast:31 into rows 2 and 3
  return v;
}

// OR of v over aligned runs of G consecutive lanes (G = 1, 2, 4 or 8); every
// lane of the wave must be active.
template <int G>
__device__ __forceinline__ uint32_t or_across_lanes(uint32_t v) {
  static_assert(G == 1 || G == 2 || G == 4 || G == 8, "run of 1, 2, 4 or 8 lanes");
  if (G >= 2) v |= (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, false);  // quad_perm 1,0,3,2
  if (G >= 4) v |= (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, false);  // quad_perm 2,3,0,1
  if (G >= 8) v |= (uint32_t)__shfl_xor((int)v, 4, 64);
  return v;
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
  for (int d = 32; d > 0; d >>= 1) v += __shfl_xor(v, d, 64);
  return v;
}

// ---------------------------------------------------------------- ticket

struct Ticket {
  uint32_t tile;  // 0-based tile index within this launch
  uint64_t seq;   // global sequence number of this tile (mod 2^40)
};

// Called by one thread of the block.
__device__ __forceinline__ uint64_t draw_ticket(uint64_t* ws) {
  return __hip_atomic_fetch_add(ws + kWordTicket, 1ull, __ATOMIC_RELAXED,
                                __HIP_MEMORY_SCOPE_AGENT);
}

// Called by one thread per block after its last draw.  The acquire-release
// increment orders every block's draws before the reset done by the last one.
__device__ __forceinline__ void finish_launch(uint64_t* ws, uint64_t g0, uint32_t ntiles,
                                              uint32_t nblocks) {
  const uint64_t d =
      __hip_atomic_fetch_add(ws + kWordDone, 1ull, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
  if (d == nblocks - 1) {
    __hip_atomic_store(ws + kWordDone, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(ws + kWordTicket, ((g0 + ntiles) & kSeqMask) << kTicketBits,
                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// A ticket value whose tile field is past any launch: "no tile".
constexpr uint64_t kNoTicket = kTicketMask;

// Tiles per ticket.  A chunk's tiles are processed in consecutive iterations,
// so the chunk's last aggregate appears kChunk - 1 iterations after its first;
// with kChunk <= RES + 1 later tiles never wait for it at resolution time.
constexpr uint32_t kChunk = 4;

// Tiles whose loads a block keeps in flight: while a block computes tile T(i),
// the loads of T(i + 1) .. T(i + kAhead) are outstanding.  A tile is 90 KiB
// of input at the default shape; one CU needs well over 100 KiB in flight to
// cover the HBM latency under full load.
constexpr int kAhead = 2;
// LDS ring of tickets: T(i) lives in slot i mod kTkRing.  Compute waves read
// slots i and i + kAhead in iteration i while the scan wave fills i + kAhead + 1.
constexpr int kTkRing = kAhead + 2 <= 4 ? 4 : 8;
static_assert(kAhead >= 1 && kAhead + 2 <= kTkRing, "ticket ring too small");
// (kernels may keep fewer tiles in flight: any AHEAD in [1, kAhead] fits the ring)

// Ticket word of tile `tile` of the launch whose first tile has sequence g0.
__device__ __forceinline__ uint64_t make_ticket(uint64_t g0, uint32_t tile, uint32_t ntiles) {
  return tile < ntiles ? ((g0 << kTicketBits) | tile) : kNoTicket;
}

__device__ __forceinline__ Ticket decode_ticket(uint64_t c) {
  Ticket tk;
  tk.tile = (uint32_t)(c & kTicketMask);
  tk.seq = ((c >> kTicketBits) + tk.tile) & kSeqMask;
  return tk;
}

// T(i) from the LDS ticket ring, as a wave-uniform (scalar) value, so that
// the tensor lookup and the per-tile bookkeeping stay out of vector registers.
__device__ __forceinline__ Ticket ticket_at(const uint64_t* s_tk, int i) {
  const uint64_t c = s_tk[i & (kTkRing - 1)];
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)c);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(c >> 32));
  return decode_ticket(((uint64_t)hi << 32) | lo);
}

// ---------------------------------------------------------------- look-back
//
// Computes the exclusive prefix of tile `tk` (tile > 0) after it has published
// its aggregate: the inclusive prefix of the nearest predecessor that has
// published one, plus the aggregates of the tiles in between.  A window of
// 64 * LK predecessors is read at once (lane i, slot m inspects tile
// j - (m*64 + i)) and consumed only when every tile up to the nearest prefix
// is ready.  The first window is issued early by the caller (look_back_issue)
// so its latency overlaps other work.  If a needed tile is not ready, only
// lane 0 polls that tile's word, with a growing pause, before the window is
// read again: device-scope loads bypass the per-XCD L2 caches, and hundreds
// of waves re-reading whole windows would flood the memory side.  The wait
// ends because tickets are handed out in order: every predecessor belongs to
// a block that is already running, and tile 0 always publishes a prefix.
template <int LK>
struct LookWindow {
  uint64_t w[LK];
};

// STRIDE: sequence numbers per tile.  A tile that runs several chained scans
// gives each its own sequence number (scan c of tile t: base + STRIDE * t +
// c); its look-back then visits the predecessors' words of the same scan.
template <int LK, int STRIDE = 1>
__device__ __forceinline__ void look_back_issue(uint64_t* ws, const Ticket& tk, int64_t j,
                                                LookWindow<LK>& win) {
  const int lane = lane_id();
#pragma unroll
  for (int m = 0; m < LK; ++m) {
    const int64_t tj = j - (m * 64 + lane);
    win.w[m] = 0;
    if (tj >= 0) {
      const uint64_t gj =
          (tk.seq - (uint64_t)STRIDE * (uint64_t)((int64_t)tk.tile - tj)) & kSeqMask;
      win.w[m] = __hip_atomic_load(status_slot(ws, gj), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// WIDE: the aggregates may exceed 32 bits (a packed multi-field value); they
// are then summed with 64-bit lane shuffles.
template <int LK, bool WIDE = false, int STRIDE = 1>
__device__ uint64_t look_back(uint64_t* ws, const Ticket& tk, LookWindow<LK> win) {
  const int lane = lane_id();
  uint64_t excl = 0;
  int64_t j = (int64_t)tk.tile - 1;
  uint32_t polls = 0;
  for (;;) {
    uint64_t pm[LK], xm[LK];
#pragma unroll
    for (int m = 0; m < LK; ++m) {
      const int64_t tj = j - (m * 64 + lane);
      const uint64_t gj =
          (tk.seq - (uint64_t)STRIDE * (uint64_t)((int64_t)tk.tile - tj)) & kSeqMask;
      if (tj >= 0 && ((win.w[m] >> 54) & 0xFFull) != ((gj >> kSlotBits) & 0xFFull))
        win.w[m] = 0;  // stale lap: not ready
      const uint64_t flag = win.w[m] >> 62;
      pm[m] = __ballot(tj >= 0 && flag == kFlagPrefix);
      xm[m] = __ballot(tj >= 0 && flag == 0);
    }
    // nearest prefix in window order (m, then lane)
    int first_m = LK, first_l = 64;
#pragma unroll
    for (int m = LK - 1; m >= 0; --m)
      if (pm[m]) { first_m = m; first_l = __builtin_ctzll(pm[m]); }
    // nearest tile that is needed but not ready
    int wait_q = -1;
#pragma unroll
    for (int m = LK - 1; m >= 0; --m) {
      uint64_t need;
      if (m < first_m) need = ~0ull;
      else if (m == first_m) need = first_l >= 63 ? ~0ull : ((2ull << first_l) - 1);
      else need = 0;
      if (xm[m] & need) wait_q = m * 64 + __builtin_ctzll(xm[m] & need);
    }
    if (wait_q >= 0) {
      // wait for that one tile, then read the window again
      const int64_t tq = j - wait_q;
      const uint64_t gq =
          (tk.seq - (uint64_t)STRIDE * (uint64_t)((int64_t)tk.tile - tq)) & kSeqMask;
      uint32_t pause = 0;
      bool ready = false;
      bool gave_up = false;
      while (!ready && !gave_up) {
        if (lane == 0) {
          const uint64_t x =
              __hip_atomic_load(status_slot(ws, gq), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          ready = (x >> 62) != 0 && ((x >> 54) & 0xFFull) == ((gq >> kSlotBits) & 0xFFull);
          // once any wave of the device has given up, nobody waits any more
          // (checked every 64th poll: the flag is only a safety net)
          if (!ready && (++polls >= kMaxPolls ||
                         ((polls & 63) == 0 &&
                          __hip_atomic_load(ws + kWordGaveUp, __ATOMIC_RELAXED,
                                            __HIP_MEMORY_SCOPE_AGENT))))
            gave_up = true;
        }
        ready = __shfl(ready ? 1 : 0, 0, 64) != 0;
        gave_up = __shfl(gave_up ? 1 : 0, 0, 64) != 0;
        if (!ready && !gave_up) {
          if (pause < 8) ++pause;
          for (uint32_t z = 0; z < pause; ++z) __builtin_amdgcn_s_sleep(2);
        }
      }
      if (!ready) {
        // gave up: only a workspace that was not zero-filled gets here
        if (lane == 0)
          __hip_atomic_store(ws + kWordGaveUp, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return excl;
      }
      look_back_issue<LK, STRIDE>(ws, tk, j, win);
      continue;
    }
    // Every word before the nearest prefix is a tile aggregate (a count of at
    // most one tile, so 64 * LK of them fit 32 bits): sum them with the DPP
    // scan instead of 64-bit lane shuffles, and take the one prefix value
    // from its lane.
    if (WIDE) {
      uint64_t a = 0;
#pragma unroll
      for (int m = 0; m < LK; ++m) {
        const bool take = m < first_m || (m == first_m && lane < first_l);
        if (take) a += win.w[m] & kValueMask;
      }
      excl += wave_sum_u64(a);
    } else {
      uint32_t a = 0;
#pragma unroll
      for (int m = 0; m < LK; ++m) {
        const bool take = m < first_m || (m == first_m && lane < first_l);
        if (take) a += (uint32_t)(win.w[m] & kValueMask);
      }
      excl += __builtin_amdgcn_readlane(wave_incl_scan(a), 63);
    }
    if (first_m < LK) {
      uint64_t pw = 0;
#pragma unroll
      for (int m = 0; m < LK; ++m)
        if (m == first_m) pw = win.w[m] & kValueMask;
      const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)pw, first_l);
      const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(pw >> 32), first_l);
      return excl + (((uint64_t)hi << 32) | lo);
    }
    j -= 64 * LK;
    look_back_issue<LK, STRIDE>(ws, tk, j, win);
  }
}

// Owner of a tile.  Lane k of a wave holds tile_begin[k] for k < ntensors
// (<= 64 tensors per launch) and ~0 elsewhere; the tensor that owns tile t is
// the highest lane whose begin is <= t (begins never decrease, and an empty
// tensor shares its begin with the next tensor, which wins).  One compare and
// one ballot, no memory access on the way.
template <typename Params>
__device__ __forceinline__ uint32_t owner_lane_begin(const Params& p) {
  uint32_t v = ~0u;
  const int lane = lane_id();
#pragma unroll
  for (int k = 0; k < 64; ++k)
    if (k < p.ntensors && lane == k) v = p.tile_begin[k];
  return v;
}

__device__ __forceinline__ int owner_of(uint32_t lane_begin, uint32_t t) {
  const uint64_t b = __ballot(lane_begin <= t);  // lane 0 holds 0 <= t
  return 63 - __builtin_clzll(b);
}

// ---------------------------------------------------------------- scan wave
//
// The loop run by the one scan wave of a persistent encode/sparsify block.
// Blocks synchronise once per iteration.  Tile T(i) is the tile whose data
// the compute waves turn into wave totals in iteration i (its loads were
// issued during iteration i - kAhead).  For each tile:
//   iteration i            compute waves publish its wave totals
//                          (s_wtot[i & 1]); after the barrier the scan wave
//                          combines them (group-major) into s_wexcl (ring
//                          of wexcl_ring(RES))
//                          and publishes the tile aggregate (tile 0 of the
//                          launch publishes its inclusive prefix, folding in
//                          the append position *count);
//   iteration i + RES      the scan wave resolves the tile: the first
//                          look-back window is read before the barrier,
//                          overlapping the compute, and is consumed after it;
//                          it publishes the inclusive prefix and stores the
//                          exclusive prefix in s_excl[i & 1];
//   iteration i + RES + 1  after the barrier the compute waves write its
//                          entries to the patch.
// Iterations from a tile's compute to its resolution (RES) and to its
// write-out (RES + 1), per kernel; a deeper lag finds more predecessors
// already resolved and costs LDS for what waits to be written.
// Ring of per-wave exclusive prefixes: filled at i, read at i + RES + 1.
constexpr int wexcl_ring(int res) {
  return res + 2 <= 4 ? 4 : res + 2 <= 8 ? 8 : res + 2 <= 16 ? 16 : 32;
}

struct ScanState {
  Ticket tk;
  uint64_t agg;
  int k;
  bool valid;
  bool ovf;  // some wave-group of the tile found more than seg_cap entries
};

// Optional outputs for encode (all null for the sparsifier):
//   s_cnt2 / s_ovf2: on resolving a tile the scan wave also stores its entry
//     count and whether one of its wave-groups found more than seg_cap entries
//     (the compaction segments overflowed);
//   s_known: the latest tile this block has resolved and its inclusive prefix,
//     two slots, slot i & 1 written in iteration i (and read by the compute
//     waves in iteration i + 2).  Entries of any later tile t lie below
//     incl + (t - tile) * tile_elems.  Before the first resolution it holds
//     (kNoTile, *count).
struct KnownPrefix {
  uint64_t incl;
  uint32_t tile;
};
constexpr uint32_t kNoTile = 0xFFFFFFFFu;

template <int U, int NW, int RES, typename Params, int AHEAD = kAhead>
__device__ void scan_wave_loop(const Params& p, uint64_t* s_tk, uint32_t* s_wtot2,
                               uint32_t* s_wexcl, uint64_t* s_excl2, uint32_t* s_cnt2,
                               uint32_t* s_ovf2, uint32_t seg_cap, KnownPrefix* s_known) {
  constexpr int kResolve = RES;
  constexpr int kDefer = RES + 1;
  constexpr int kWexclRing = wexcl_ring(RES);
  static_assert(kChunk <= kDefer, "a chunk's tiles must all be computed before the first resolves");
  const int lane = lane_id();
  // tiles come in chunks of kChunk consecutive tiles, one atomic per chunk;
  // next_tile / left: the unused part of the block's current chunk.  The next
  // chunk is always drawn one chunk ahead (`pre`, lane 0), so the atomic's
  // round trip overlaps a whole chunk of iterations instead of delaying the
  // ticket store that the compute waves wait for at the barrier.
  uint64_t g0 = 0, pre = 0;
  uint32_t next_tile = 0, left = 0;
  auto take = [&]() -> uint64_t {  // lane 0 only
    if (left == 0) {
      const uint64_t c = pre;
      pre = draw_ticket(p.ws);
      g0 = c >> kTicketBits;
      next_tile = (uint32_t)(c & kTicketMask) * kChunk;
      left = kChunk;
    }
    --left;
    return make_ticket(g0, next_tile++, p.ntiles);
  };
  if (lane == 0) {
    if (s_known) {
      const uint64_t c0 = __hip_atomic_load(p.count, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      s_known[0] = KnownPrefix{c0, kNoTile};
      s_known[1] = KnownPrefix{c0, kNoTile};
    }
    pre = draw_ticket(p.ws);
    bool more = true;
    for (int q = 0; q <= AHEAD; ++q) {
      s_tk[q] = more ? take() : kNoTicket;
      more = decode_ticket(s_tk[q]).tile < p.ntiles;
    }
  }
  __syncthreads();  // T(0) .. T(AHEAD)
  // g0 (lane 0 only) comes from the counter itself: a ticket slot may hold
  // kNoTicket when the block's first chunk lies past the last tile, and the
  // sequence base must never move backwards
  uint64_t count_in = 0;
  const uint32_t lane_begin = owner_lane_begin(p);
  ScanState hist[kDefer];  // hist[d]: T(i - 1 - d)
#pragma unroll
  for (int d = 0; d < kDefer; ++d) hist[d].valid = false;
  for (int it = 0;; ++it) {
    const Ticket cur = ticket_at(s_tk, it);
    const bool have_cur = cur.tile < p.ntiles;
    bool pending = have_cur;
#pragma unroll
    for (int d = 0; d < kDefer; ++d) pending |= hist[d].valid;
    if (!pending) break;
    const bool have_last = ticket_at(s_tk, it + AHEAD).tile < p.ntiles;
    if (lane == 0) s_tk[(it + AHEAD + 1) & (kTkRing - 1)] = have_last ? take() : kNoTicket;
    // first look-back window of T(i - kResolve), overlapping the compute of T(i)
    const ScanState res = hist[kResolve - 1];
    LookWindow<kLookK> win;
    const bool walk = res.valid && res.tk.tile != 0;
    if (walk) look_back_issue<kLookK>(p.ws, res.tk, (int64_t)res.tk.tile - 1, win);
    __syncthreads();  // wave totals of T(i) are in s_wtot[i & 1]; T(i + AHEAD + 1) in s_tk
    ScanState now;
    now.valid = have_cur;
    if (have_cur) {
      const uint32_t v = lane < U * NW ? s_wtot2[(it & 1) * U * NW + lane] : 0u;
      const uint32_t incl = wave_incl_scan(v);
      if (lane < U * NW) s_wexcl[(it & (kWexclRing - 1)) * U * NW + lane] = incl - v;
      now.tk = cur;
      now.agg = __shfl(incl, 63, 64);
      now.ovf = __ballot(lane < U * NW && v > seg_cap) != 0;
      now.k = owner_of(lane_begin, cur.tile);
      if (cur.tile == 0) {
        count_in = *p.count;  // append position, written by an earlier call
        if (lane == 0) status_publish(p.ws, cur.seq, kFlagPrefix, count_in + now.agg);
      } else if (lane == 0) {
        status_publish(p.ws, cur.seq, kFlagAggregate, now.agg);
      }
    }
    if (res.valid) {
      uint64_t excl;
      if (!walk) {
        excl = count_in;
      } else {
        excl = look_back<kLookK>(p.ws, res.tk, win);
        if (lane == 0) status_publish(p.ws, res.tk.seq, kFlagPrefix, excl + res.agg);
      }
      if (lane == 0) {
        s_excl2[(it - kResolve) & 1] = excl;
        if (s_cnt2) s_cnt2[(it - kResolve) & 1] = (uint32_t)res.agg;
        if (s_ovf2) s_ovf2[(it - kResolve) & 1] = res.ovf ? 1u : 0u;
        if (s_known) s_known[it & 1] = KnownPrefix{excl + res.agg, res.tk.tile};
        if (res.tk.tile == p.ntiles - 1) *p.count = excl + res.agg;
        if (p.seg_begin) {
          // segment starts of this tensor and of the empty tensors just before it
          if (p.tile_begin[res.k] == res.tk.tile) {
            for (int kk = res.k; kk >= 0 && p.tile_begin[kk] == res.tk.tile; --kk)
              p.seg_begin[kk] = excl;
          }
          // empty tensors at the end of the batch start where the patch ends
          if (res.tk.tile == p.ntiles - 1) {
            for (int kk = res.k + 1; kk < p.ntensors; ++kk) p.seg_begin[kk] = excl + res.agg;
          }
        }
      }
    }
    if (s_known && !res.valid && lane == 0) s_known[it & 1] = s_known[(it - 1) & 1];
#pragma unroll
    for (int d = kDefer - 1; d > 0; --d) hist[d] = hist[d - 1];
    hist[0] = now;
  }
  if (lane == 0) finish_launch(p.ws, g0, p.ntiles, gridDim.x);
}

// ---------------------------------------------------------------- loads

__device__ __forceinline__ uint4 load16(const void* p) {
  return *reinterpret_cast<const uint4*>(p);
}

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

// 16-byte load with the non-temporal hint: streamed data that is read once
// should not displace what the caches hold.
__device__ __forceinline__ uint4 load16_stream(const void* p) {
  const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ void store16_stream(void* p, uint4 v) {
  u32x4_t w;
  w.x = v.x; w.y = v.y; w.z = v.z; w.w = v.w;
  __builtin_nontemporal_store(w, reinterpret_cast<u32x4_t*>(p));
}

__device__ __forceinline__ void store16(void* p, uint4 v) {
  *reinterpret_cast<uint4*>(p) = v;
}

// Scalar stores and loads with the non-temporal hint.  The patch and the
// refreshed lines are written once and not read again by this pass; with the
// hint, interleaving those writes with the streamed reads costs HBM time
// close to their byte count (measured on the 32B-shaped set: the whole-line
// refresh 2.2 ms and the patch 0.5 ms cheaper per step than plain stores).
template <typename T>
__device__ __forceinline__ void store_nt(T* p, T v) {
  __builtin_nontemporal_store(v, p);
}

template <typename T>
__device__ __forceinline__ T load_nt(const T* p) {
  return __builtin_nontemporal_load(p);
}

__device__ __forceinline__ uint32_t get_u32(const uint4& v, int i) {
  return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w;
}


// Blocks of `kernel` (launched with `block` threads) that fit on the current
// device at once: the grid of a persistent launch.  The occupancy query is
// made once per (device, kernel) and remembered.
inline int persistent_grid(const void* kernel, int block) {
  struct Entry {
    const void* kernel;
    int dev, block, grid;
  };
  static Entry cache[64];
  static int used = 0;
  static std::mutex mu;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  {
    std::lock_guard<std::mutex> g(mu);
    for (int i = 0; i < used; ++i)
      if (cache[i].kernel == kernel && cache[i].dev == dev && cache[i].block == block)
        return cache[i].grid;
  }
  int cus = 0, per_cu = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, block, 0) != hipSuccess) return 0;
  int grid = cus * (per_cu > 0 ? per_cu : 1);
  if (grid > (int)kMaxGrid) grid = (int)kMaxGrid;
  std::lock_guard<std::mutex> g(mu);
  if (used < 64) cache[used++] = Entry{kernel, dev, block, grid};
  return grid;
}

}  // namespace pulse
