"""CPU oracle of the policy-masked MoE layer (test infrastructure only; see pmpe_oracle)."""
