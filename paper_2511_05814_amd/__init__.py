"""MI355X-native MoE decode under expert offloading.

The compute path lives in the HIP library built from `csrc/` and is reached
through `paper_2511_05814_amd.binding` (ctypes over the C ABI declared in
`include/moe_offload.h`).  `workload` generates the seeded synthetic inputs.
Importing the package does not load the library; `binding.lib()` does, and it
raises if the library has not been built.
"""
