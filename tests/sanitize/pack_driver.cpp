// Drives the host packers of libqx under the sanitizers: for each case on the command
// line (bits kind group n k seed) it draws codes and tables with a small LCG, packs them
// with qx_pack_layout or qx_pack_q4x (rows >= 256 take the multithreaded path), and
// writes the blob to <out_dir>/<index>.bin; it also exercises the error paths.
#include <cstdio>
#include <cstdlib>
#include <string>
#include <vector>

#include "../../include/qx.h"

static uint32_t lcg(uint64_t& s) {
  s = s * 6364136223846793005ull + 1442695040888963407ull;
  return (uint32_t)(s >> 33);
}

int main(int argc, char** argv) {
  if (argc < 3) return 2;
  const std::string out = argv[1];
  int bad = 0;
  for (int i = 2; i + 5 < argc + 1; i += 6) {
    const int bits = atoi(argv[i]), kind = atoi(argv[i + 1]), group = atoi(argv[i + 2]);
    const int n = atoi(argv[i + 3]), k = atoi(argv[i + 4]);
    uint64_t s = strtoull(argv[i + 5], nullptr, 10);
    const qx_desc d = {n, k, bits, group, kind, 0};
    const size_t nk = (size_t)n * k, G = (size_t)k / group;
    std::vector<uint8_t> codes(nk);
    for (auto& c : codes) c = (uint8_t)(lcg(s) % (1u << bits));
    size_t size = 0;
    int st;
    std::vector<uint8_t> blob;
    if (kind == QX_Q4X) {
      std::vector<uint16_t> scales(n * G), cb(64);
      std::vector<uint8_t> sel(n * G);
      for (auto& v : scales) v = (uint16_t)(0x3000 + lcg(s) % 0x1000);
      for (auto& v : sel) v = (uint8_t)(lcg(s) % 4);
      for (auto& v : cb) v = (uint16_t)(lcg(s) & 0xBBFF);
      st = qx_pack_q4x(&d, codes.data(), scales.data(), sel.data(), cb.data(), nullptr, 0, &size);
      blob.assign(size, 0xCD);
      if (st == QX_OK) st = qx_pack_q4x(&d, codes.data(), scales.data(), sel.data(), cb.data(), blob.data(), size, &size);
      if (size > 0 && qx_pack_q4x(&d, codes.data(), scales.data(), sel.data(), cb.data(), blob.data(), size - 1, &size) != QX_E_SIZE) ++bad;
    } else if (kind == QX_UNIFORM) {
      std::vector<uint16_t> scales(n * G), zeros(n * G);
      for (auto& v : scales) v = (uint16_t)(0x1800 + lcg(s) % 0x1000);
      static const uint16_t kZeros[8] = {0x0000, 0x3C00, 0x4000, 0x4200, 0x4400, 0x4500, 0x4600, 0x4700};
      for (auto& v : zeros) v = kZeros[lcg(s) % 8];
      st = qx_pack_layout(&d, codes.data(), scales.data(), zeros.data(), nullptr, nullptr, 0, &size);
      blob.assign(size, 0xCD);
      if (st == QX_OK) st = qx_pack_layout(&d, codes.data(), scales.data(), zeros.data(), nullptr, blob.data(), size, &size);
      if (n > 0) {
        zeros[0] = 0x3800;  // 0.5: not an integer
        if (qx_pack_layout(&d, codes.data(), scales.data(), zeros.data(), nullptr, blob.data(), size, &size) != QX_E_ARG) ++bad;
      }
    } else {
      std::vector<uint16_t> cb(n * G << bits);
      for (auto& v : cb) v = (uint16_t)(lcg(s) & 0xBBFF);
      st = qx_pack_layout(&d, codes.data(), nullptr, nullptr, cb.data(), nullptr, 0, &size);
      blob.assign(size, 0xCD);
      if (st == QX_OK) st = qx_pack_layout(&d, codes.data(), nullptr, nullptr, cb.data(), blob.data(), size, &size);
      if (n > 0) {
        codes[nk - 1] = (uint8_t)(1u << bits);  // out of range
        if (qx_pack_layout(&d, codes.data(), nullptr, nullptr, cb.data(), blob.data(), size, &size) != QX_E_ARG) ++bad;
      }
    }
    if (st != QX_OK) { fprintf(stderr, "case %d: status %d\n", i / 6, st); return 1; }
    FILE* f = fopen((out + "/" + std::to_string(i / 6) + ".bin").c_str(), "wb");
    if (!f) return 3;
    if (!blob.empty()) fwrite(blob.data(), 1, blob.size(), f);
    fclose(f);
  }
  // descriptor errors reach no packer
  const qx_desc bad_desc = {4, 100, 3, 64, QX_UNIFORM, 0};
  size_t sz;
  if (qx_pack_layout(&bad_desc, nullptr, nullptr, nullptr, nullptr, nullptr, 0, &sz) != QX_E_ARG) ++bad;
  if (qx_gemv(&bad_desc, nullptr, nullptr, nullptr, nullptr) != QX_E_ARG) ++bad;
  printf("sanitized packer: %d unexpected statuses\n", bad);
  return bad ? 4 : 0;
}
