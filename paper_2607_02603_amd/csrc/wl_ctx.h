// Shared structures of the device path: the per-call device state, the
// pointer bundle every kernel receives, and the tuning constants.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wl {

constexpr int kBlock = 256;          // threads per workgroup (4 waves)
constexpr uint32_t kSmallMax = 2048; // class/bucket size sorted in LDS
constexpr uint32_t kTinyMax = 64;    // class/bucket size sorted in one wave
constexpr uint32_t kMidMax = 512;    // ... sorted by one wave in LDS (counting sort)
constexpr uint32_t kPicoMax = 8;     // ... sorted by 8 lanes (kept at the back of the tiny list)
constexpr uint32_t kTile = 2048;     // elements per tile in the MSD passes
constexpr uint32_t kTilePerThread = kTile / kBlock;
constexpr int kRadixBits = 8;
constexpr int kRadix = 1 << kRadixBits;
constexpr int kPasses = 8;           // 61-bit keys: 7 passes of 8 bits + 5
constexpr uint32_t kMatBit = 0x80000000u;  // small segment keys are in 'keys'
constexpr uint32_t kHeavyChunk = 4096;     // entries per heavy-row chunk
constexpr int kNumBins = 4;                // row-length bins of the SpMV
constexpr int kScanBlocks = 1024;          // blocks of the device-wide scans
constexpr uint32_t kTableMax = 65535;      // largest k of the compact gathers

// Kinds of image launches (diagnostics): gathering SpMV, propagation
// blocking, one-colour rounds.
constexpr int kImgGather = 0, kImgPb = 1, kImgUniform = 2;

// Row-length bins of the SpMV: lanes per row.
//   bin 0: len <= 8        4 lanes
//   bin 1: len <= 64      16 lanes
//   bin 2: len <= 4096    64 lanes (one wave)
//   bin 3: len  > 4096    chunks of kHeavyChunk entries, one wave each
__host__ __device__ __forceinline__ int row_bin(uint64_t len) {
  return len <= 8 ? 0 : (len <= 64 ? 1 : (len <= kHeavyChunk ? 2 : 3));
}

// Device-resident scalars of one call.
struct DevState {
  uint32_t k;           // colour count before the current round
  uint32_t k_new;       // colour count after it
  uint32_t round;       // index of the round to run next
  uint32_t done;        // 0 running, 1 stable, 2 round cap reached, 3 and 4 halted for
                        // the host (wl_relabel.h), 5 stopped on an error (err)
  uint32_t max_rounds;  // stop after this many rounds in total
  uint32_t n_small;     // entries in the small-segment list
  uint32_t err;         // input errors seen on the device (bit mask)
  uint32_t n_chunks;    // heavy-row chunks of the SpMV schedule
  uint32_t bin_cnt[kNumBins];
  uint32_t bin_start[kNumBins];
  uint32_t n_tiny;      // entries in the tiny-segment list (<= 64 nodes)
  uint32_t dense;       // 1 if the colours in use are exactly [0, k)
  uint32_t n_live;      // live classes (wl_live.h) of the current round
  uint32_t nl;          // their members
  uint32_t n_live2;     // the same for the next round
  uint32_t nl2;
  uint32_t nsub;        // sub-classes of the live classes after the sort
  uint32_t nosplit;     // 1 when no live class split in this round
  uint32_t n_split;     // live classes that split
  uint32_t split_any;   // 1 when some live class split in this round
  uint32_t shift_big;   // 1 when the splits need the per-colour shift table
  uint32_t max_deg;     // largest row length (saturated at 2^32 - 1)
  uint32_t deg_nd;      // distinct row lengths (one-colour round)
  uint32_t n_mid;       // live rows queued for one wave each (this round)
  uint32_t n_hlive;     // live heavy rows (this round)
  uint32_t n_pico;      // segments of <= kPicoMax nodes (this round)
  uint32_t n_msort;     // segments of kTinyMax + 1 .. kMidMax nodes (this round)
  uint32_t tickets[4];  // chunk tickets of this round's chained scans (per site)
  uint64_t seed;
  // The two big-segment lists: (entries << 32) | tiles.  One 64-bit atomic
  // appends a segment and reserves its tiles, so the tile offsets come out
  // in list order without a scan.
  unsigned long long big[2];
  unsigned long long work[3][2];    // diagnostics: rows, entries per image kind
  unsigned long long act_entries;   // entries of the rows whose image is needed
  unsigned long long sym_hash[2];   // validation: hashes of (i, j) and (j, i)
};

struct HeavyChunk {
  uint64_t beg;   // first entry
  uint32_t len;   // entries (<= kHeavyChunk)
  uint32_t row;   // node
  uint32_t h;     // index of the heavy row (accumulator slot)
  uint32_t nc;    // chunks of that row
};

// Block ranges of the single SpMV launch: [0, heavy) heavy chunks,
// [heavy, b2) one wave per row, [b2, b1) 16 lanes per row, [b1, b0) 4 lanes.
struct SpmvGrid {
  uint32_t heavy, b2, b1, b0;
};

// Every pointer a kernel may touch.  Passed by value.
struct Ctx {
  uint32_t n;
  uint64_t nnz;
  const uint32_t* rp32;
  const uint64_t* rp64;
  const uint32_t* col;
  const uint32_t* wgt;
  DevState* st;
  uint32_t* c;         // colours, node order
  uint64_t* x;         // scratch of the quotient phase (8 bytes per node)
  uint64_t* wtab;      // per-colour random values (k <= 65535)
  uint16_t* c16;       // compact colours (k <= 65535)
  uint8_t* c8;         // compact colours (k <= 255)
  uint64_t* z;         // image A x
  uint32_t* perm;      // nodes grouped by colour (positions)
  uint32_t* perm_tmp;
  uint64_t* keys;      // z in position order (big segments)
  uint64_t* keys_tmp;
  uint8_t* flags;      // 1 where a new (colour, z) group starts
  uint8_t* act;        // 1 if the node's row needs an image (full relabel); in the
                       // incremental rounds: 1 for heavy rows of live classes
  uint32_t* ids;       // inclusive scan of flags minus one
  uint32_t* cstart;    // class c occupies perm[cstart[c] .. cstart[c+1])
  uint2* small_list;   // (start, len | kMatBit), kMidMax < len <= kSmallMax from the
                       // front, kTinyMax < len <= kMidMax from the back
  uint2* tiny_list;    // (start, len | kMatBit), 2 <= len <= 64
  uint2* big_list0;
  uint2* big_list1;
  uint32_t* tile_off0; // first tile of every segment of big_list0 (list order)
  uint32_t* tile_off1; // the same for big_list1
  uint32_t* bhist;     // per (big segment, bucket)
  unsigned long long* bmin;
  unsigned long long* bmax;
  uint32_t* bcur;
  uint32_t* scan_part; // kScanBlocks partial sums
  uint32_t* rows;      // SpMV bin lists, concatenated
  uint32_t* bin_part;  // kNumBins * kScanBlocks
  HeavyChunk* chunks;
  unsigned long long* hacc;  // two accumulators per heavy row
  uint32_t* hcnt;            // finished chunks per heavy row
  uint32_t max_small, max_big, max_chunks, max_heavy;
  uint32_t max_sm;     // capacity of small_list (the mid segments fill it from the back)
  int weighted;
  uint32_t ring;       // 0: image in F_p (p = 2^61 - 1); 1: in Z/2^64 (wl_device.h)
  int nt_stream;       // stream col_idx with non-temporal loads
  uint32_t cs_fix;     // largest mixed bucket the small-segment sort fixes by insertion
  uint32_t chain_spins;  // polls a chained scan waits for an earlier chunk before it gives up
  // Batch mode (Algorithm 2): the rows are nodes [ext_lo, ext_lo + n) of a
  // larger graph; a column outside that range is a node frozen as its own
  // singleton class, whose value is W(seed, r, 2^32 + column).
  int batch;
  uint32_t ext_lo;
  int keys_mat;        // segment keys are already in 'keys' (no gather of z)
  // Live classes of the incremental rounds (wl_live.h).  Several of these
  // share memory with buffers of the full relabel that those rounds do not
  // use (see make_ctx).
  uint32_t* lperm;     // members of the live classes, class after class
  uint32_t* pos_deg;   // the same map as written by the one-colour round (the
                       // same buffer; kept for graphs whose rounds do not keep it)
  uint32_t* pos;       // position of every node in lperm, ~0 outside the live
                       // classes (NULL outside in-core sessions)
  uint32_t* lperm2;
  uint32_t* qcls;      // live class of every position of lperm
  uint32_t* qcls2;
  uint32_t* lcold;     // colour of each live class
  uint32_t* loff;      // its first position in lperm
  uint32_t* llen;      // its size
  uint32_t* lcold2;
  uint32_t* loff2;
  uint32_t* llen2;
  uint32_t* gstart;    // per sub-class: first position
  uint32_t* gend;      // one past its last position
  uint8_t* gnz;        // 1 if it holds a non-empty row
  uint32_t* gl;        // per sub-class (or class): live flag, then its index
  uint32_t* go;        // size, then its first position
  uint2* split;        // (old colour, extra sub-classes) of the classes that split
  uint32_t* shift;     // per colour: extra sub-classes below it (many splits)
  uint64_t* rs;        // per position of lperm: first entry of its node's row
  uint64_t* rs2;
  uint32_t* rl;        // and the row's length
  uint32_t* rl2;
  uint32_t* midq;      // positions whose rows get one wave each (this round)
  uint32_t* hq;        // positions with heavy rows (this round)
  uint8_t* lsplit;     // per live class: 1 if it split in this round
  uint8_t* bsame;      // per big segment of a radix pass: 1 if all its keys are equal
  unsigned long long* desc;  // chained-scan descriptors, 2 * desc_cap (NULL outside
                             // in-core sessions); cleared at the start of a call
  uint32_t desc_cap;
  uint8_t* nz0f;       // per sub-class: a member with key 0 has a non-empty row
                       // (set by k_live_scan_final, consumed and cleared by
                       // k_live_subs_splits; NULL outside in-core sessions)
};

}  // namespace wl
