"""InfiniPot-V KV-cache compression pass for AMD MI355X (gfx950).

The pass -- TaR and VaN scores, keep-set selection, in-place compaction -- is
hand-written HIP in ``csrc/`` behind the C ABI of ``include/ipv.h``;
``paper_2506_15745_amd.ipv`` is its ctypes binding for torch tensors.
"""
