// Limits and LDS layout of the Top-S sparse replay attention (paper App. C.4,
// "Post-Translation Phase: Cache Replay").  Plain constexpr C++ with no HIP
// dependency: the host-side argument check, the kernel dispatch and the
// kernel itself read the same definitions, and a host-only program can
// enumerate them.
#pragma once

#include <stddef.h>

namespace mot {

// LDS of the sparse kernel, per workgroup: V_sel^T [D][S] and P [16][S] in
// bf16, then 128 floats of cross-wave reductions.
constexpr size_t replay_sparse_lds_bytes(int D, int S) { return (size_t)(D * S + 16 * S) * 2 + 128 * sizeof(float); }
constexpr size_t kReplaySparseLdsMax = 65536;

// Largest set size each head dim is instantiated for (the register arrays of
// the kernel are sized for it).  Both fit the 64 KB LDS limit.
constexpr int replay_sparse_smax(int D) { return D == 128 ? 192 : 256; }
static_assert(replay_sparse_lds_bytes(128, replay_sparse_smax(128)) <= kReplaySparseLdsMax, "LDS of S = 192, D = 128");
static_assert(replay_sparse_lds_bytes(64, replay_sparse_smax(64)) <= kReplaySparseLdsMax, "LDS of S = 256, D = 64");

// Set sizes the sparse kernel accepts: a multiple of 32 from 32 up to the
// instantiated maximum of the head dim (D = 64 or 128).
constexpr bool replay_sparse_supported(int D, int S) {
    return (D == 64 || D == 128) && S >= 32 && S % 32 == 0 && S <= replay_sparse_smax(D) &&
           replay_sparse_lds_bytes(D, S) <= kReplaySparseLdsMax;
}

// XOR swizzle of the LDS rows of S keys (SC = S / 8 sixteen-byte chunks per
// row): chunk c of row d is stored at c ^ (d & mask).  The mask comes from
// the largest power of two (at most 16) that divides SC, so the permuted
// chunk stays inside the row for every SC.
constexpr int replay_swizzle_mask(int sc) { return ((sc & -sc) < 16 ? (sc & -sc) : 16) - 1; }

// The instantiation that serves a set of S keys: sets of up to 128 keys use
// the kernel sized for 128 (fewer registers, more waves per SIMD), larger
// sets the one sized for the maximum of the head dim.
constexpr int replay_sparse_instance(int D, int S) { return S <= 128 ? 128 : replay_sparse_smax(D); }

// Per-thread item counts of the kernel for sets of up to SMAX keys (256
// threads, four waves): V key-pair items of 16 bytes, and 16-key blocks of
// the score product per wave.  Both round up.
constexpr int replay_sparse_v_items(int D, int smax) { return ((smax / 2) * (D / 8) + 255) / 256; }
constexpr int replay_sparse_key_blocks(int smax) { return (smax / 16 + 3) / 4; }

// The two-position form of the sparse kernel: the union of two sets of up to
// 128 keys, with the 2G query heads of the pair as the 16 columns of the
// score product.
constexpr bool replay_sparse_pair_supported(int D, int S, int G) {
    return replay_sparse_supported(D, S) && S <= 128 && G >= 1 && 2 * G <= 16;
}

// The full causal kernel addresses a batch row's K (and V^T) through 32-bit
// byte offsets: rows of `ts` elements (H_kv * D for BTHD, D for BHTD) for
// T positions must stay under 2 GiB.
constexpr bool replay_causal_supported(long long T, long long H_kv, int D, bool bthd) {
    return (T + 64) * (bthd ? H_kv * D : D) * 2 < (1LL << 31);
}

}  // namespace mot
