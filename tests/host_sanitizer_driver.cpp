// Host-code driver for the sanitizer test (tests/test_host_sanitizers.py).
//
// Built with -fsanitize=address,undefined together with the library's host
// code (wc_host.cpp: analysis, encoder, blob parsing) and the oracle (its own
// object, declared here).  The driver:
//   - encodes seeded tensors of every dtype (byte runs, row-major and
//     column-block tiles, per-tensor and layer codebooks, 64 and 32 lanes,
//     several chunk sizes, edge sizes) with wc_encode and with the oracle, and
//     requires byte-identical blobs;
//   - decodes each blob with the oracle and requires the original bytes;
//   - re-opens each blob with wc_open, then opens truncated copies and copies
//     with flipped bytes, which must be refused or accepted without any
//     sanitizer report (the decode of an accepted corrupt blob is the GPU's);
//   - runs wc_analyze on every tensor.
// Exit status 0 when every check holds; the sanitizers abort on any error.
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <vector>

#include "../include/wc.h"

extern "C" {
typedef struct {
  const uint8_t* data;
  uint64_t nbytes;
  uint32_t dtype;
  uint64_t rows, cols;
} orc_tensor;
int orc_encode_blob(const orc_tensor* ts, uint32_t n_tensors, uint32_t chunk_bytes, uint32_t L,
                    uint32_t tile_r, uint32_t tile_c, uint32_t tile_order, uint32_t shared_tables,
                    uint8_t** blob_out, uint64_t* size_out);
int orc_decode_blob(const uint8_t* b, uint64_t size, uint8_t* const* outs);
void orc_free(void* p);
}

namespace {

uint64_t rng = 0x9E3779B97F4A7C15ull;
uint32_t next() {  // xorshift64*
  rng ^= rng >> 12;
  rng ^= rng << 25;
  rng ^= rng >> 27;
  return uint32_t((rng * 0x2545F4914F6CDD1Dull) >> 32);
}

// Skewed bytes (most mass near a few values), so the tables are not flat.
std::vector<uint8_t> draw(uint64_t n, int dtype) {
  std::vector<uint8_t> v(n);
  for (uint64_t i = 0; i < n; i++) {
    const uint32_t r = next();
    const uint32_t sym = (r & 7) == 0 ? (r >> 8) & 0xFF : (r >> 8) % 9 + 120;
    v[i] = uint8_t(sym);
  }
  if (dtype == WC_BF16 || dtype == WC_FP16)  // low bytes near-uniform (mantissa)
    for (uint64_t i = 0; i < n; i += 2) v[i] = uint8_t(next());
  return v;
}

int failures = 0;
void fail(const char* what, int c) {
  fprintf(stderr, "case %d: %s\n", c, what);
  failures++;
}

struct Case {
  int dtype;
  uint64_t rows, cols;  // symbol elements; rows = 0: a byte run of `bytes`
  uint64_t bytes;
  uint32_t chunk, lanes, tile_r, tile_c, order, layer;
};

uint64_t bytes_of(int dtype, uint64_t rows, uint64_t cols) {
  const uint64_t n = rows * cols;
  return dtype == WC_BF16 || dtype == WC_FP16 ? 2 * n : (dtype == WC_U4 || dtype == WC_FP4_E2M1 ? n / 2 : n);
}

void run(const Case& k, int c) {
  // two tensors of the case's dtype plus one bf16 byte run, so layer codebooks
  // and several descriptors are exercised
  const uint64_t nb = k.rows ? bytes_of(k.dtype, k.rows, k.cols) : k.bytes;
  std::vector<std::vector<uint8_t>> data = {draw(nb, k.dtype), draw(nb, k.dtype), draw(998, WC_BF16)};
  wc_tensor wt[3];
  orc_tensor ot[3];
  for (int t = 0; t < 3; t++) {
    const int dt = t < 2 ? k.dtype : WC_BF16;
    const uint64_t r = t < 2 ? k.rows : 0, cl = t < 2 ? k.cols : 0;
    wt[t] = wc_tensor{data[t].data(), data[t].size(), dt, 0, r, cl};
    ot[t] = orc_tensor{data[t].data(), data[t].size(), uint32_t(dt), r, cl};
  }
  wc_params p{k.chunk, k.lanes, 12, 4, k.tile_r, k.tile_c, k.layer, k.order};
  wc_blob* b = nullptr;
  if (wc_encode(wt, 3, &p, &b) != WC_OK) {
    fail("wc_encode", c);
    return;
  }
  uint8_t* ob = nullptr;
  uint64_t osz = 0;
  if (orc_encode_blob(ot, 3, k.chunk, k.lanes, k.tile_r, k.tile_c, k.order, k.layer, &ob, &osz)) {
    fail("orc_encode_blob", c);
  } else {
    if (osz != b->size || memcmp(ob, b->data, osz)) fail("blobs differ", c);
    std::vector<std::vector<uint8_t>> outs(3);
    uint8_t* ptrs[3];
    for (int t = 0; t < 3; t++) {
      outs[t].assign(data[t].size() + 1, 0xAB);
      ptrs[t] = outs[t].data();
    }
    if (orc_decode_blob(ob, osz, ptrs)) fail("oracle decode", c);
    for (int t = 0; t < 3; t++)
      if (!data[t].empty() && memcmp(outs[t].data(), data[t].data(), data[t].size()))
        fail("round trip", c);
    orc_free(ob);
  }
  // re-open the blob, then truncated and corrupted copies
  std::vector<uint8_t> bytes(b->data, b->data + b->size);
  wc_blob* o = nullptr;
  if (wc_open(bytes.data(), bytes.size(), &o) != WC_OK) fail("wc_open", c);
  else wc_free(o);
  for (uint64_t cut : {uint64_t(0), uint64_t(16), bytes.size() / 2, bytes.size() - 1}) {
    o = nullptr;
    if (wc_open(bytes.data(), cut, &o) == WC_OK) {
      fail("truncated blob accepted", c);
      wc_free(o);
    }
  }
  for (int f = 0; f < 64; f++) {
    std::vector<uint8_t> bad = bytes;
    const uint64_t at = f < 32 ? next() % std::min<uint64_t>(bad.size(), 1024) : next() % bad.size();
    bad[at] ^= uint8_t(1u << (next() & 7));
    o = nullptr;
    if (wc_open(bad.data(), bad.size(), &o) == WC_OK) wc_free(o);  // either outcome, no report
  }
  for (int t = 0; t < 3; t++) {
    wc_stats st;
    if (wc_analyze(&wt[t], &st) != WC_OK) fail("wc_analyze", c);
  }
  wc_free(b);
}

}  // namespace

int main() {
  std::vector<Case> cases;
  const int dts[] = {WC_BF16, WC_FP16, WC_U8, WC_U4, WC_FP8_E4M3, WC_FP8_E5M2, WC_FP4_E2M1};
  for (int dt : dts) {
    for (uint32_t lanes : {64u, 32u})
      for (uint64_t n : {uint64_t(0), uint64_t(2), uint64_t(4094), uint64_t(65538)})
        cases.push_back({dt, 0, 0, n, 4096, lanes, 0, 0, 0, 0});
    for (uint32_t order : {0u, 1u})
      for (uint32_t layer : {0u, 1u})
        cases.push_back({dt, 128, 512, 0, 8192, 64, 16, 256, order, layer});
    cases.push_back({dt, 64, 1024, 0, 65536, 64, 64, 512, 1, 0});
    cases.push_back({dt, 96, 256, 0, 4096, 32, 32, 128, 0, 1});   // row-major 32 x 128 tiles
    cases.push_back({dt, 100, 256, 0, 4096, 64, 32, 128, 1, 0});  // tile does not divide: flat
  }
  int c = 0;
  for (const Case& k : cases) run(k, c++);
  printf("%d cases, %d failures\n", c, failures);
  return failures ? 1 : 0;
}
