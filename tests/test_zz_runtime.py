"""The library and torch must share one HIP runtime in the process."""


def test_single_hip_runtime_loaded():
    import paper_2107_02103_amd.binding  # noqa: F401
    import torch  # noqa: F401
    maps = open("/proc/self/maps").read()
    hip = {line.split()[-1] for line in maps.splitlines() if "libamdhip64" in line}
    assert len(hip) == 1, hip
