"""MI355X-native hot path of TGL (Zhou et al., VLDB 2022): T-CSR build and
multi-hop temporal neighbour sampling, and the feature / state lookup of the
sampled slots, as hand-written HIP kernels behind the C
ABI of include/tgl.h.  ``binding`` marshals torch tensors into that ABI;
``workloads`` draws the seeded synthetic graphs and root streams."""
from .binding import (TCSR, Hop, Sampler, TglError, lib, sample, sample_capacity,  # noqa: F401
                      status_str, tcsr_build, tcsr_build_workspace, tcsr_from_host, tcsr_from_columns, tcsr_columns,
                      pack_entries, timer_enable, timer_disable, timer_read, timer_reset, timer_select,
                      gather, time_encode, pointers_reset, mfg_export, MFG, EXPORTS, LIB_PATH, MOST_RECENT, UNIFORM, KEY_NODE, KEY_EDGE)
