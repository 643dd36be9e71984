// numa.h -- binding the calling thread to the NUMA node of a PCI device (internal
// to the library; host only, Linux sysfs and system calls, no HIP).  App. B binds
// the generation process to the NUMA node that owns the GPU's PCIe root, so that
// pinned host memory for reloads sits next to the device.
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace omnimem {

// Parses a sysfs CPU list ("0-3,8,10-11") into bits of `mask` (mask_words 64-bit
// words).  Returns the number of CPUs set, or -1 on a malformed list or a CPU
// beyond the mask.
int parse_cpu_list(const char* text, uint64_t* mask, int mask_words);

// NUMA node of PCI device `bus_id` ("0000:c1:00.0", any letter case) read under
// sysfs_root ("/sys" on a live system): >= 0, or -1 when the system reports none.
int numa_node_of_pci(const char* sysfs_root, const char* bus_id);

// Binds the calling thread to node `node`: its CPU affinity becomes the node's
// CPUs that it may already run on, and its memory policy prefers the node (pinned
// host buffers it allocates afterwards are placed there).  Threads it starts
// later inherit both.  Returns 0 when bound, 1 when nothing was changed (the node
// shares no CPU with the current affinity), -1 on a failed read or system call.
int bind_thread_to_node(const char* sysfs_root, int node);

}  // namespace omnimem
