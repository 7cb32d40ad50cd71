// The transfer path driven through the C ABI alone: no Python, no torch.
// Device memory comes from hipMalloc and the stream from hipStreamCreate.
//
// Two block-major pools (3 layers, block size 16, 2 KV heads, head_dim 64,
// fp16: 4 KiB chunks, 24 KiB blocks).  The sender's allocator uses the
// segment policy on a pool with every fifth block held; the receiver's uses a
// seeded shuffled free list.  Request A (30 blocks) is planned, its plan
// copied to the device and moved with flowkv_transfer; request B (12 blocks)
// is moved with flowkv_transfer_inline from the host plan; request C (10
// blocks) is planned and moved in one flowkv_transfer_request call.  Two
// error paths are checked on the way.
//
// Writes to <out_dir>: src.bin (the sender pool), dst_before.bin and
// dst_after.bin (the receiver pool around the two transfers) and tables.txt
// (geometry and run counts, then the sender and receiver block lists of A, B
// and C).  A test
// compares dst_after with the oracle's result on src and dst_before.
// Prints "abi ok" and exits 0 when every call returned what it should.
//
// Usage: abi_transfer <out_dir>
#include <hip/hip_runtime_api.h>

#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <string>
#include <vector>

#include "flowkv.h"

namespace {

constexpr int32_t kLayers = 3, kBlockSize = 16, kKvHeads = 2, kHeadDim = 64, kElem = 2;
constexpr int64_t kChunk = int64_t(kBlockSize) * kKvHeads * kHeadDim * kElem;  // 4 KiB
constexpr int64_t kBlock = 2 * kLayers * kChunk;                                 // 24 KiB
constexpr int32_t kSrcBlocks = 96, kDstBlocks = 80;

[[noreturn]] void die(const char* what, const char* detail) {
  std::fprintf(stderr, "abi_transfer: %s: %s\n", what, detail);
  std::exit(1);
}

void hip_ok(hipError_t e, const char* what) {
  if (e != hipSuccess) die(what, hipGetErrorString(e));
}

void fk_ok(int rc, const char* what) {
  if (rc != FLOWKV_OK) die(what, flowkv_last_error());
}

// splitmix64 (Steele, Lea & Flood 2014), for the pools' seeded contents
uint64_t next(uint64_t& s) {
  uint64_t z = (s += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

std::vector<uint8_t> seeded_bytes(size_t n, uint64_t seed) {
  std::vector<uint8_t> v(n);
  for (size_t i = 0; i < n; i += 8) {
    const uint64_t x = next(seed);
    for (size_t k = 0; k < 8 && i + k < n; ++k) v[i + k] = uint8_t(x >> (8 * k));
  }
  return v;
}

void write_file(const std::string& path, const void* data, size_t n) {
  FILE* f = std::fopen(path.c_str(), "wb");
  if (!f || std::fwrite(data, 1, n, f) != n) die("write", path.c_str());
  std::fclose(f);
}

void write_list(FILE* f, const char* name, const std::vector<int32_t>& v) {
  std::fprintf(f, "%s", name);
  for (int32_t x : v) std::fprintf(f, " %d", x);
  std::fprintf(f, "\n");
}

std::vector<flowkv_segment> plan(const std::vector<int32_t>& S, const std::vector<int32_t>& D) {
  // first with too small a capacity: ECAP, and n_out gives the need
  int64_t need = 0;
  flowkv_segment one{};
  const int rc = flowkv_plan(S.data(), D.data(), int32_t(S.size()), kSrcBlocks, kDstBlocks, &one,
                             0, &need);
  if (need > 0 && rc != FLOWKV_ECAP) die("flowkv_plan", "capacity 0 was accepted");
  std::vector<flowkv_segment> segs(size_t(need > 0 ? need : 1));
  int64_t n = 0;
  fk_ok(flowkv_plan(S.data(), D.data(), int32_t(S.size()), kSrcBlocks, kDstBlocks, segs.data(),
                    int64_t(segs.size()), &n),
        "flowkv_plan");
  if (n != need) die("flowkv_plan", "run count differs from the reported need");
  segs.resize(size_t(n));
  return segs;
}

}  // namespace

int main(int argc, char** argv) {
  if (argc != 2) {
    std::fprintf(stderr, "usage: abi_transfer <out_dir>\n");
    return 2;
  }
  const std::string dir = argv[1];
  const size_t src_bytes = size_t(kSrcBlocks) * kBlock, dst_bytes = size_t(kDstBlocks) * kBlock;

  // pools
  void* src_dev = nullptr;
  void* dst_dev = nullptr;
  hip_ok(hipMalloc(&src_dev, src_bytes), "hipMalloc sender pool");
  hip_ok(hipMalloc(&dst_dev, dst_bytes), "hipMalloc receiver pool");
  const std::vector<uint8_t> src_host = seeded_bytes(src_bytes, 11);
  const std::vector<uint8_t> dst_before = seeded_bytes(dst_bytes, 12);
  hip_ok(hipMemcpy(src_dev, src_host.data(), src_bytes, hipMemcpyHostToDevice), "upload sender");
  hip_ok(hipMemcpy(dst_dev, dst_before.data(), dst_bytes, hipMemcpyHostToDevice),
         "upload receiver");
  void* src_base[1] = {src_dev};
  void* dst_base[1] = {dst_dev};
  const flowkv_pool src{FLOWKV_LAYOUT_BLOCK_MAJOR, kLayers, kSrcBlocks, 0, kChunk, src_base};
  const flowkv_pool dst{FLOWKV_LAYOUT_BLOCK_MAJOR, kLayers, kDstBlocks, 0, kChunk, dst_base};

  // allocators: a fragmented sender pool, a shuffled receiver free list
  flowkv_allocator* sa = nullptr;
  flowkv_allocator* da = nullptr;
  fk_ok(flowkv_allocator_create(kSrcBlocks, FLOWKV_POLICY_SEGMENT, 0, &sa), "sender allocator");
  fk_ok(flowkv_allocator_create(kDstBlocks, FLOWKV_POLICY_FIFO_SHUFFLED, 7, &da),
        "receiver allocator");
  std::vector<int32_t> held;
  for (int32_t b = 0; b < kSrcBlocks; b += 5) held.push_back(b);
  fk_ok(flowkv_mark_used(sa, held.data(), int32_t(held.size())), "flowkv_mark_used");
  std::vector<int32_t> SA(30), DA(30), SB(12), DB(12), SC(10), DC(10);
  fk_ok(flowkv_alloc(sa, 30, SA.data()), "alloc sender A");
  fk_ok(flowkv_alloc(da, 30, DA.data()), "alloc receiver A");
  fk_ok(flowkv_alloc(sa, 12, SB.data()), "alloc sender B");
  fk_ok(flowkv_alloc(da, 12, DB.data()), "alloc receiver B");
  fk_ok(flowkv_alloc(sa, 10, SC.data()), "alloc sender C");
  fk_ok(flowkv_alloc(da, 10, DC.data()), "alloc receiver C");

  hipStream_t stream;
  hip_ok(hipStreamCreate(&stream), "hipStreamCreate");

  // request A: plan in device memory
  const std::vector<flowkv_segment> pa = plan(SA, DA);
  void* segs_dev = nullptr;
  hip_ok(hipMalloc(&segs_dev, pa.size() * sizeof(flowkv_segment)), "hipMalloc plan");
  hip_ok(hipMemcpy(segs_dev, pa.data(), pa.size() * sizeof(flowkv_segment),
                   hipMemcpyHostToDevice),
         "upload plan");
  if (flowkv_transfer(nullptr, &dst, static_cast<const flowkv_segment*>(segs_dev),
                      int64_t(pa.size()), 30, stream) != FLOWKV_EINVAL)
    die("flowkv_transfer", "a NULL sender pool was accepted");
  fk_ok(flowkv_transfer(&src, &dst, static_cast<const flowkv_segment*>(segs_dev),
                        int64_t(pa.size()), 30, stream),
        "flowkv_transfer");

  // request B: plan in the kernel arguments
  const std::vector<flowkv_segment> pb = plan(SB, DB);
  fk_ok(flowkv_transfer_inline(&src, &dst, pb.data(), int64_t(pb.size()), 12, nullptr, stream),
        "flowkv_transfer_inline");

  // request C: planned and launched in one call
  int64_t runs_c = -1;
  fk_ok(flowkv_transfer_request(&src, &dst, SC.data(), DC.data(), 10, nullptr, &runs_c, stream),
        "flowkv_transfer_request");

  hip_ok(hipStreamSynchronize(stream), "hipStreamSynchronize");
  std::vector<uint8_t> dst_after(dst_bytes);
  hip_ok(hipMemcpy(dst_after.data(), dst_dev, dst_bytes, hipMemcpyDeviceToHost),
         "download receiver");

  write_file(dir + "/src.bin", src_host.data(), src_bytes);
  write_file(dir + "/dst_before.bin", dst_before.data(), dst_bytes);
  write_file(dir + "/dst_after.bin", dst_after.data(), dst_bytes);
  FILE* f = std::fopen((dir + "/tables.txt").c_str(), "w");
  if (!f) die("write", "tables.txt");
  std::fprintf(f, "%d %d %d %d %d %zu %zu %lld\n", kLayers, kBlockSize,
               kKvHeads * kHeadDim * kElem, kSrcBlocks, kDstBlocks, pa.size(), pb.size(),
               (long long)runs_c);
  write_list(f, "SA", SA);
  write_list(f, "DA", DA);
  write_list(f, "SB", SB);
  write_list(f, "DB", DB);
  write_list(f, "SC", SC);
  write_list(f, "DC", DC);
  std::fclose(f);

  hip_ok(hipStreamDestroy(stream), "hipStreamDestroy");
  hip_ok(hipFree(segs_dev), "hipFree plan");
  hip_ok(hipFree(src_dev), "hipFree sender pool");
  hip_ok(hipFree(dst_dev), "hipFree receiver pool");
  flowkv_allocator_destroy(sa);
  flowkv_allocator_destroy(da);
  std::printf("abi ok: %zu, %zu and %lld runs moved\n", pa.size(), pb.size(), (long long)runs_c);
  return 0;
}
