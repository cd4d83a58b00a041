"""The build refuses a library whose kernels spill registers to scratch."""

def test_build_rejects_kernels_that_spill():
    from paper_2508_02751_amd.build import scratch_users
    remarks = ("x.hip:1:1: remark: Function Name: kern_a [-Rpass-analysis=kernel-resource-usage]\n"
               "x.hip:1:1: remark:     ScratchSize [bytes/lane]: 0 [-Rpass]\n"
               "x.hip:9:1: remark: Function Name: kern_b [-Rpass-analysis=kernel-resource-usage]\n"
               "x.hip:9:1: remark:     ScratchSize [bytes/lane]: 48 [-Rpass]\n")
    assert scratch_users(remarks) == [("kern_b", 48)]
