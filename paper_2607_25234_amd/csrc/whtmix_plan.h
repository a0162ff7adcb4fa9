// Plan table shared by the host entry points and the kernel launchers.
//
// The mixer of one slice is, on the flattened row-major index f = n*C + c of
// length L = N*C = 2^K, y = (1/L) H_L (g o H_L x) with H_L the +/-1 Sylvester
// matrix: H_N (x) H_C = H_{N*C} in Sylvester order, so the channel and token
// transforms of section III-B (eqs. (2)-(3)) together are one Walsh-Hadamard
// transform over all K bits of f, and the four 1/sqrt factors multiply to 1/L.
// Sylvester butterflies over disjoint bit groups commute and need no twiddle
// factors, so any split of the K bits into passes is exact.
#pragma once

namespace whtmix {

enum PlanKind {
    PLAN_AUTO = 0,
    PLAN_SMALL = 1,
    PLAN_FUSED = 2,
    PLAN_THREE_PASS = 3,
    PLAN_ONE_LAUNCH = 4,
    PLAN_WAVE_TILES = 5,
    PLAN_TWO_PASS = 6
};

constexpr int kMaxLog2Slice = 30;   // N*C <= 2^30
constexpr int kMaxSmall = 10;       // SMALL: L <= 2^10
constexpr int kMinTile = 11;        // tiles hold 2^11 .. 2^15 elements
constexpr int kMaxTile = 15;
// FUSED (one workgroup per slice): up to 2^16 elements, as two 2^15 register
// sets above 2^15 (the mixer's forward; the backward pass and the block run
// the three-pass plan for 2^16-element slices).  One workgroup moves a 2^16
// slice in about 23 us whatever the batch, so AUTO takes it from 48 slices,
// where the three passes (15 us at 16 slices, 24 us at 48) stop being faster.
constexpr int kMaxFused = 16;
constexpr int kFusedPairMinBatch = 48;

// Wave tiles (whtmix_wave.hip): the three passes of slices of 2^12 .. 2^16
// elements on one-wave 2^9-element tiles, as three launches (WAVE_TILES) or
// one (ONE_LAUNCH, passes ordered by per-slice completion counters).  x and
// y move in 16-byte groups, so a slice's element count must be a multiple
// of 8.  ONE_LAUNCH's counter block holds 2B + 3 words (per-slice counters
// of two passes, exits, the call's error word, the sticky error word), so it
// takes at most kOneLaunchMaxBatch slices.
constexpr int kWaveMinK = 12;
constexpr int kWaveMaxK = 16;
// AUTO takes WAVE_TILES for slices of 2^16 elements up to 3 slices (measured
// crossover against THREE_PASS).
constexpr int kWave16MaxBatch = 3;
// TWO_PASS (whtmix_wave.hip): a fold pass in place of passes 1 and 2, then
// pass 3; slices of 2^15 and 2^16 elements.  AUTO takes it for 2^15-element
// slices up to 48 (one launch fewer than WAVE_TILES, and from 17 slices
// faster than one workgroup per slice until about 48) and for 2^16-element
// slices from 4 (after WAVE_TILES) up to 16 (then THREE_PASS): measured
// faster there with x in cache and with x from memory.  Up to 3 slices of
// 2^16 a fold workgroup's 256 KiB read (float32) from memory costs about the
// launch it saves.
constexpr int kTwoPassMinK = 15;
constexpr int kTwoPass15MaxBatch = 48;
constexpr int kTwoPass16MaxBatch = 16;
constexpr int kCounterWords = 4096;
constexpr int kOneLaunchMaxBatch = (kCounterWords - 3) / 2;
// Polls of a ONE_LAUNCH wait before it gives up (about a second or two).
constexpr unsigned kDefaultSpinLimit = 1u << 21;

// Forward middle pass: slices per workgroup.  A workgroup takes one run in nb
// slices in turn and reads the run's gain once.  nb doubles while it divides
// B and the grid keeps at least kMiddleMinWaves waves (16 per CU, a full
// round of the 2^14-element tiles); stereo64k (4 slices of 2^23) gets 4:
// its middle pass 51.2 -> 48.9 us.  run_bits = A - R, thread_bits = the
// log2 of the workgroup size.
constexpr long long kMiddleMinWaves = 4096;
constexpr long long middle_slices_per_group(long long B, int run_bits, int thread_bits)
{
    const long long waves = thread_bits > 6 ? 1ll << (thread_bits - 6) : 1ll;
    long long nb = 1;
    while (B % (2 * nb) == 0 && (B / (2 * nb)) * (1ll << run_bits) * waves >= kMiddleMinWaves)
        nb *= 2;
    return nb;
}

// whtmix_forward_noalloc: the fixed device scratch (32 MiB of floats) that
// holds its three-pass workspace, B * N_pad * C floats at most.
constexpr long long kNoAllocScratchFloats = 1ll << 23;

// THREE_PASS split for slice bits K:
//   outer passes: contiguous chunks of 2^A elements (all A low bits of f);
//   middle pass : the HB = K - A high bits, for a run of 2^R contiguous low
//                 elements carried along (R bits untransformed), so one middle
//                 tile holds 2^(HB + R) elements.
struct Split {
    int A, HB, R;
};

constexpr int clampi(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }

// Automatic split for K >= 16: balance the outer and middle tile sizes and
// carry runs of 32 floats (128 bytes) where the tile limits allow.
constexpr Split auto_split(int K)
{
    int A = clampi((K + 6) / 2, kMinTile, kMaxTile);
    int HB = K - A;
    int R = clampi(5, kMinTile - HB, kMaxTile - HB);
    return Split{A, HB, R};
}

// Forced THREE_PASS for 12 <= K <= 15 (the shapes FUSED would take).
constexpr Split forced_split(int K)
{
    return Split{kMinTile, K - kMinTile, 2 * kMinTile - K};
}

// Split of the block's three-pass kernels (projections fused into the outer
// passes, whose tiles stay within 2^15 elements).
constexpr Split module_split(int K)
{
    return K >= 16 ? auto_split(K) : forced_split(K);
}

// Split with outer tiles of 2^16 (two 2^15 register sets per workgroup),
// K >= 17.
constexpr int kMaxOuter = 16;
constexpr Split pair_split(int K)
{
    const int HB = K - kMaxOuter;
    return Split{kMaxOuter, HB, clampi(5, kMinTile - HB, kMaxTile - HB)};
}

// Split of the mixer's three-pass kernels.  Slices of 2^26 elements and more
// take outer tiles of 2^16, which leaves the middle pass one more carried
// bit: runs of 32 floats (128-byte lines) at 2^26 instead of 16.
constexpr Split three_pass_split(int K)
{
    return K < 26 ? module_split(K) : pair_split(K);
}

// The block with C = 2^8 channels (bf16) takes 2^16 outer tiles at every
// three-pass size: a tile of 256 tokens gives each wave 16 whole rows, the
// shape of the 16-row matrix-core operands.
constexpr int kPairModuleCbits = 8;
constexpr int kPairModuleMinK = 17;

}  // namespace whtmix
