"""CPU oracle (test infrastructure only: tests, smoke check and the bench's CPU baseline)."""
from . import onmt_oracle
