// numa.cpp -- NUMA node of a PCI device and binding of the calling thread to it
// (host only; Linux).
#include "numa.h"

#include <ctype.h>
#include <sched.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include <sys/syscall.h>
#include <unistd.h>

namespace omnimem {
namespace {

constexpr int kMaxCpus = 4096;
constexpr int kMaskWords = kMaxCpus / 64;
constexpr int kMpolPreferred = 1;  // MPOL_PREFERRED of the set_mempolicy system call

// Reads at most cap-1 bytes of a small sysfs file; false if it cannot be read.
bool read_small_file(const char* path, char* buf, size_t cap) {
  FILE* f = fopen(path, "r");
  if (f == nullptr) return false;
  const size_t got = fread(buf, 1, cap - 1, f);
  fclose(f);
  buf[got] = '\0';
  return got > 0;
}

}  // namespace

int parse_cpu_list(const char* text, uint64_t* mask, int mask_words) {
  if (text == nullptr || mask == nullptr || mask_words < 1) return -1;
  memset(mask, 0, sizeof(uint64_t) * static_cast<size_t>(mask_words));
  const int limit = mask_words * 64;
  int count = 0;
  const char* p = text;
  while (*p != '\0' && *p != '\n') {
    if (!isdigit(static_cast<unsigned char>(*p))) return -1;
    char* end = nullptr;
    const long lo = strtol(p, &end, 10);
    long hi = lo;
    p = end;
    if (*p == '-') {
      ++p;
      if (!isdigit(static_cast<unsigned char>(*p))) return -1;
      hi = strtol(p, &end, 10);
      p = end;
    }
    if (lo < 0 || hi < lo || hi >= limit) return -1;
    for (long c = lo; c <= hi; ++c) {
      uint64_t& w = mask[c / 64];
      const uint64_t bit = uint64_t{1} << (c % 64);
      if (!(w & bit)) ++count;
      w |= bit;
    }
    if (*p == ',') {
      ++p;
      if (*p == '\0' || *p == '\n') return -1;
    } else if (*p != '\0' && *p != '\n') {
      return -1;
    }
  }
  return count;
}

int numa_node_of_pci(const char* sysfs_root, const char* bus_id) {
  if (sysfs_root == nullptr || bus_id == nullptr) return -1;
  char id[64];
  size_t n = 0;
  for (; bus_id[n] != '\0' && n + 1 < sizeof(id); ++n) id[n] = static_cast<char>(tolower(bus_id[n]));
  id[n] = '\0';
  if (n == 0 || bus_id[n] != '\0' || strchr(id, '/') != nullptr) return -1;
  char path[512];
  if (snprintf(path, sizeof(path), "%s/bus/pci/devices/%s/numa_node", sysfs_root, id) >= static_cast<int>(sizeof(path)))
    return -1;
  char buf[32];
  if (!read_small_file(path, buf, sizeof(buf))) return -1;
  char* end = nullptr;
  const long node = strtol(buf, &end, 10);
  if (end == buf || node < 0 || node > 4095) return -1;
  return static_cast<int>(node);
}

int bind_thread_to_node(const char* sysfs_root, int node) {
  if (sysfs_root == nullptr || node < 0 || node >= kMaxCpus) return -1;
  char path[512];
  if (snprintf(path, sizeof(path), "%s/devices/system/node/node%d/cpulist", sysfs_root, node) >=
      static_cast<int>(sizeof(path)))
    return -1;
  char buf[4096];
  if (!read_small_file(path, buf, sizeof(buf))) return -1;
  uint64_t node_cpus[kMaskWords];
  if (parse_cpu_list(buf, node_cpus, kMaskWords) < 0) return -1;
  cpu_set_t now;
  CPU_ZERO(&now);
  if (sched_getaffinity(0, sizeof(now), &now) != 0) return -1;
  cpu_set_t want;
  CPU_ZERO(&want);
  int shared = 0;
  for (int c = 0; c < kMaxCpus && c < CPU_SETSIZE; ++c)
    if (((node_cpus[c / 64] >> (c % 64)) & 1u) && CPU_ISSET(c, &now)) {
      CPU_SET(c, &want);
      ++shared;
    }
  if (shared == 0) return 1;
  if (sched_setaffinity(0, sizeof(want), &want) != 0) return -1;
  uint64_t nodes[kMaskWords] = {};
  nodes[node / 64] = uint64_t{1} << (node % 64);
  if (syscall(SYS_set_mempolicy, kMpolPreferred, nodes, static_cast<unsigned long>(kMaxCpus + 1)) != 0) return -1;
  return 0;
}

}  // namespace omnimem
