"""Consumer side of the IPC handoff test (run as its own process by
tests/test_gpu_ipc.py): map the buffer another process loaded, build the
tensor views at base + offset from an index-only handle, and check every
tensor against the generator's bytes."""

import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402
import torch  # noqa: E402

from paper_2401_14351_amd import binding, synth  # noqa: E402


def main() -> int:
    ckpt_dir, desc_hex, workload = sys.argv[1:4]
    print("[ipc-consumer] importing", flush=True)
    stream = torch.cuda.Stream()
    imp = binding.Import(bytes.fromhex(desc_hex), stream)
    buf = imp.tensor()
    with binding.Checkpoint(ckpt_dir, index_only=True) as ck:
        tensors = ck.tensors()
    views = binding.views(buf, tensors)
    spec = synth.config(workload)
    with torch.cuda.stream(stream):  # ordered after the exporter's load event
        got = [views[t.name].contiguous().view(torch.uint8).cpu().numpy().reshape(-1) for t in spec.tensors]
    stream.synchronize()
    for i, (t, g) in enumerate(zip(spec.tensors, got)):
        if not np.array_equal(g, synth.tensor_bytes(spec, i)):
            print(f"[ipc-consumer] tensor {t.name} differs", flush=True)
            return 1
    del views, buf
    imp.close()
    # a descriptor whose range runs past the shared allocation is refused
    # before anything could read it
    bad = binding.IpcDesc.from_buffer_copy(bytes.fromhex(desc_hex))
    bad.offset = bad.offset + bad.bytes
    try:
        binding.Import(bytes(bad), stream)
    except binding.SllmError as e:
        if e.code != -1:
            print(f"[ipc-consumer] an out-of-range descriptor gave {e}", flush=True)
            return 1
    else:
        print("[ipc-consumer] an out-of-range descriptor was accepted", flush=True)
        return 1
    print(f"ipc ok {len(tensors)} tensors", flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
